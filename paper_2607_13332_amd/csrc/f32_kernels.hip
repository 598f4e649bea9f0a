// Stage-boundary codec with float32 storage on the matrix cores:
// v_mfma_f32_16x16x4_f32 multiplies float32 operands and accumulates in
// float32, so no operand is split.  Paper: section 4.1, Eq. (2) --
// Z = (X - E[ids]) U, X' = E[ids] + Z U^T; the gradient forms are the same
// kernels without the embedding.
//
// Both kernels walk d in 64-wide chunks (256 contiguous bytes of a float32
// row) and stage the chunk's 64 rows of U [d, K] (K = 16, 32, .., 128 floats
// per row) once per block into a row-major LDS tile of pitch K + 4 floats,
// double buffered, one barrier per chunk.  Activation and embedding rows
// travel as 4 rows x 256 contiguous bytes per instruction.
#include "ssn_device.h"
#include "ssn_launch.h"

#include <type_traits>

namespace ssn {

// 16x16x4 float32 MFMA.  A (16 x 4): lane l holds row l%16, K element l/16;
// B (4 x 16): lane l holds column l%16, K element l/16; C (16 x 16): lane l
// holds rows 4 (l/16) .. +3 of column l%16.  Only the pairing of K elements
// between A and B matters, so each kernel picks the index a K slot carries.
__device__ __forceinline__ f32x4 mfma16x16x4f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

constexpr int kF32Chunk = 64;

bool f32_uses_mfma(int64_t d, int64_t k) {
  return d % kF32Chunk == 0 && d <= INT32_MAX && k % 16 == 0 && k >= 16 && k <= 128;
}

// U rows [64 c, 64 c + 64) of U [d, K] are one contiguous span of 64 K
// floats; thread tid stages its 16-byte pieces p = tid + T i into the LDS tile
// (row 4p / K, column 4p % K, pitch K + 4).  Threads past the last piece load
// the last piece again and do not store it.
template <int K, int T>
struct UStage {
  static constexpr int UP = K + 4;
  static constexpr int NP = kF32Chunk * K / 4;
  static constexpr int FPT = (NP + T - 1) / T;
  int src[FPT], dst[FPT];
  bool on[FPT];
  __device__ __forceinline__ explicit UStage(int tid) {
#pragma unroll
    for (int i = 0; i < FPT; ++i) {
      const int p0 = tid + T * i;
      on[i] = NP % T == 0 || p0 < NP;
      const int p = on[i] ? p0 : NP - 1;
      src[i] = 4 * p;
      dst[i] = (4 * p / K) * UP + (4 * p) % K;
    }
  }
  __device__ __forceinline__ void load(const float* __restrict__ U, int c, f32x4 (&r)[FPT]) const {
    const float* base = U + (int64_t)c * kF32Chunk * K;
#pragma unroll
    for (int i = 0; i < FPT; ++i) r[i] = *(const f32x4*)(base + src[i]);
  }
  __device__ __forceinline__ void store(float* tile, const f32x4 (&r)[FPT]) const {
#pragma unroll
    for (int i = 0; i < FPT; ++i)
      if (on[i]) *(f32x4*)(tile + dst[i]) = r[i];
  }
};

// ===========================================================================
// decompress / gradient expansion.  Output tiles are computed transposed,
// Y^T [16 d x 16 tokens] = U_rows [16 d x 4] . Z^T [4 x 16 tokens]; MFMA
// (q, s) pairs K slot g with coordinate 16 q + 4 g + s, so a lane's A values
// for s = 0..3 are one 16-byte LDS read of a U row and its B values four
// coordinates of its token, held in registers for the whole kernel.  Lane
// (token n16, g) then holds d = 16 tt + 4 g .. + 3 of its token for tile tt:
// parked in a wave-private XOR-swizzled LDS tile, read back as row pieces,
// E[ids] added (loaded one chunk ahead), stored non-temporally.  Block = 8
// waves x 16 tokens; with fewer tokens than fill the chip a second grid
// dimension splits d (decompress_grid_split).  Tokens past N recompute token
// N - 1 and store the same bytes there.  GZ: the coordinate row of token t is
// Z[ids[t]] (a gathered table), with no embedding added.
// ===========================================================================
template <int KQ, bool HAS_E, bool GZ>
__global__ __launch_bounds__(512) void decompress_f32_mfma(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids, const float* __restrict__ E,
    const float* __restrict__ U, float* __restrict__ Y, int64_t N, int d, int64_t V,
    const uint16_t* __restrict__ Zb, int kz) {
  static_assert(!(HAS_E && GZ), "gathered coordinates carry no additive embedding");
  constexpr int K = 16 * KQ, DC = kF32Chunk, W = 8;
  using Stage = UStage<K, 64 * W>;
  constexpr int UP = Stage::UP, FPT = Stage::FPT;
  __shared__ __align__(16) float ut[2][DC * UP];
  __shared__ f32x4 st[W][16 * 16];                 // [wave][token * 16 + (cell ^ token)]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = (int64_t)blockIdx.x * (16 * W) + 16 * wave;

  // B operand: coordinates 16 q + 4 g + s of token n16 (zero past kz)
  float zf[KQ][4];
  {
    int64_t t = tok0 + n16;
    t = t < N ? t : N - 1;
    const int64_t zrow = (GZ ? clamp_id(ids[t], V) : t) * (int64_t)kz;
#pragma unroll
    for (int q = 0; q < KQ; ++q)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int c = 16 * q + 4 * g + s;
        zf[q][s] = c < kz ? (Zb ? bf16_to_f32(Zb[zrow + c]) : Zc[zrow + c]) : 0.f;
      }
  }
  // epilogue rows: instruction m covers tokens 4 m .. 4 m + 3, 16 lanes each
  float* yrow[4];
  const float* erow[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    int64_t t = tok0 + 4 * m + g;
    t = t < N ? t : N - 1;
    yrow[m] = Y + t * d + 4 * n16;
    erow[m] = HAS_E ? E + clamp_id(ids[t], V) * d + 4 * n16 : nullptr;
  }
  const Stage stage(tid);
  f32x4 ust[2][FPT];
  f32x4 ering[2][4];
  auto load_e = [&](int c, f32x4(&eo)[4]) {
    if constexpr (HAS_E) {
#pragma unroll
      for (int m = 0; m < 4; ++m) eo[m] = *(const f32x4*)(erow[m] + c * DC);
    }
  };

  const int nch = d / (DC * (int)gridDim.y);
  const int pbase = (int)blockIdx.y * nch;
  const int rot = (int)(blockIdx.x % (unsigned)nch);
  auto chunk = [&](int i) {
    const int x = i + rot;
    return pbase + (x < nch ? x : x - nch);
  };
  auto last = [&](int i) { return i < nch ? i : nch - 1; };
  f32x4* sw = st[wave];

  // chunk i, i % 2 == B: loads for later chunks, barrier, MFMAs, epilogue,
  // then the LDS store of chunk i + 1's U (loaded one chunk earlier)
  auto body = [&](int i, auto Bc) {
    constexpr int B = decltype(Bc)::value;
    const int c = chunk(i);
    stage.load(U, chunk(last(i + 2)), ust[B]);
    load_e(chunk(last(i + 1)), ering[B ^ 1]);
    __syncthreads();
    const float* ub = ut[B];
    f32x4 acc[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < KQ; ++q)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const f32x4 a = *(const f32x4*)(ub + (16 * tt + n16) * UP + 16 * q + 4 * g);
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[tt] = mfma16x16x4f32(a[s], zf[q][s], acc[tt]);
      }
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) sw[n16 * 16 + ((4 * tt + g) ^ n16)] = acc[tt];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int r = 4 * m + g;
      f32x4 v = sw[r * 16 + (n16 ^ r)];
      if constexpr (HAS_E) v += ering[B][m];
      __builtin_nontemporal_store(v, (f32x4*)(yrow[m] + c * DC));
    }
    stage.store(ut[B ^ 1], ust[B ^ 1]);
  };

  stage.load(U, chunk(0), ust[0]);
  stage.load(U, chunk(last(1)), ust[1]);
  load_e(chunk(0), ering[0]);
  stage.store(ut[0], ust[0]);
  int i = 0;
  for (; i + 1 < nch; i += 2) {
    body(i, std::integral_constant<int, 0>{});
    body(i + 1, std::integral_constant<int, 1>{});
  }
  if (i < nch) body(i, std::integral_constant<int, 0>{});
}

// ===========================================================================
// compress / gradient projection, Z [N, kz] = (X - E[ids]) U (or X U, minus
// P[ids] with the projected table).  C = D [16 tokens x 4] . U [4 x 16]:
// MFMA (q, s) pairs K slot g with d = 16 q + 4 g + s, so a lane's A values
// for s = 0..3 are one 16-byte read of its token's row of D from the
// wave-private tile it was parked in (X - E formed in registers, one float32
// rounding).  Column slot j of tile i is coordinate KP j + i, so the B values
// of all KP tiles for one (q, s) are the KP contiguous floats
// U[16 q + 4 g + s][KP j ..] of the staged tile, and lane (j, g) ends with
// coordinates KP j .. KP j + KP - 1 of tokens 4 g .. 4 g + 3.  Block = W
// waves x 16 tokens, every wave sweeping all of d (start rotated per block).
// ===========================================================================
template <int KP, bool HAS_E, bool HAS_P, int W>
__global__ __launch_bounds__(64 * W) void compress_f32_mfma(
    const float* __restrict__ X, const int32_t* __restrict__ ids, const float* __restrict__ E,
    const float* __restrict__ U, float* __restrict__ Z, int64_t N, int d, int64_t V,
    const float* __restrict__ Pt, uint16_t* __restrict__ Zb, int kz) {
  static_assert(!(HAS_E && HAS_P), "the embedding is subtracted as rows or as projected rows");
  constexpr int K = 16 * KP, DC = kF32Chunk;
  using Stage = UStage<K, 64 * W>;
  constexpr int UP = Stage::UP, FPT = Stage::FPT;
  __shared__ __align__(16) float ut[2][DC * UP];
  __shared__ f32x4 dt[W][16 * 16];                 // [wave][token * 16 + (cell ^ token)]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = (int64_t)blockIdx.x * (16 * W) + 16 * wave;

  // rows: instruction m covers tokens 4 m .. 4 m + 3, 16 lanes (256 bytes) each
  const float* xrow[4];
  const float* erow[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    int64_t t = tok0 + 4 * m + g;
    t = t < N ? t : N - 1;
    xrow[m] = X + t * d + 4 * n16;
    erow[m] = HAS_E ? E + clamp_id(ids[t], V) * d + 4 * n16 : nullptr;
  }
  const Stage stage(tid);
  f32x4 ust[2][FPT];
  f32x4 xs[2][4], es[2][4];
  auto load_rows = [&](int c, f32x4(&xo)[4], f32x4(&eo)[4]) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      xo[m] = __builtin_nontemporal_load((const f32x4*)(xrow[m] + c * DC));
      if constexpr (HAS_E) eo[m] = *(const f32x4*)(erow[m] + c * DC);
    }
  };

  const int nch = d / DC;
  const int rot = (int)(blockIdx.x % (unsigned)nch);
  auto chunk = [&](int i) {
    const int x = i + rot;
    return x < nch ? x : x - nch;
  };
  auto last = [&](int i) { return i < nch ? i : nch - 1; };
  f32x4* dw = dt[wave];
  f32x4 acc[KP];
#pragma unroll
  for (int i = 0; i < KP; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto body = [&](int i, auto Bc) {
    constexpr int B = decltype(Bc)::value;
    stage.load(U, chunk(last(i + 2)), ust[B]);
    load_rows(chunk(last(i + 1)), xs[B ^ 1], es[B ^ 1]);
    // park chunk i's rows of D
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int r = 4 * m + g;
      dw[r * 16 + (n16 ^ r)] = HAS_E ? xs[B][m] - es[B][m] : xs[B][m];
    }
    __syncthreads();
    const float* ub = ut[B];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 a = dw[n16 * 16 + ((4 * q + g) ^ n16)];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const float* ur = ub + (16 * q + 4 * g + s) * UP + KP * n16;
        float b[KP];
        if constexpr (KP % 4 == 0) {
#pragma unroll
          for (int h = 0; h < KP; h += 4) {
            const f32x4 v = *(const f32x4*)(ur + h);
            b[h] = v[0]; b[h + 1] = v[1]; b[h + 2] = v[2]; b[h + 3] = v[3];
          }
        } else if constexpr (KP % 2 == 0) {
#pragma unroll
          for (int h = 0; h < KP; h += 2) {
            const f32x2 v = *(const f32x2*)(ur + h);
            b[h] = v[0]; b[h + 1] = v[1];
          }
        } else {
#pragma unroll
          for (int h = 0; h < KP; ++h) b[h] = ur[h];
        }
#pragma unroll
        for (int h = 0; h < KP; ++h) acc[h] = mfma16x16x4f32(a[s], b[h], acc[h]);
      }
    }
    stage.store(ut[B ^ 1], ust[B ^ 1]);
  };

  stage.load(U, chunk(0), ust[0]);
  load_rows(chunk(0), xs[0], es[0]);
  stage.load(U, chunk(last(1)), ust[1]);
  stage.store(ut[0], ust[0]);
  int i = 0;
  for (; i + 1 < nch; i += 2) {
    body(i, std::integral_constant<int, 0>{});
    body(i + 1, std::integral_constant<int, 1>{});
  }
  if (i < nch) body(i, std::integral_constant<int, 0>{});

  // lane (j, g): coordinates KP j + h of tokens 4 g + r
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t t = tok0 + 4 * g + r;
    if (t >= N) continue;
#pragma unroll
    for (int h = 0; h < KP; ++h) {
      const int col = KP * n16 + h;
      if (col >= kz) continue;
      float v = acc[h][r];
      if constexpr (HAS_P) v -= Pt[clamp_id(ids[t], V) * kz + col];
      if (Zb)
        Zb[t * kz + col] = (uint16_t)f32_to_bf16(v);
      else
        Z[t * kz + col] = v;
    }
  }
}

// ===========================================================================
// Launchers.
// ===========================================================================
template <int KQ>
static hipError_t launch_decompress_f32_kq(dim3 grid, int64_t N, int d, int64_t V, const float* Z,
                                           const int32_t* ids, const float* E, const float* U,
                                           float* Y, bool gather_z, hipStream_t st,
                                           const uint16_t* Zb, int kz) {
  if (E)
    hipLaunchKernelGGL((decompress_f32_mfma<KQ, true, false>), grid, dim3(512), 0, st, Z, ids, E, U,
                       Y, N, d, V, Zb, kz);
  else if (gather_z)
    hipLaunchKernelGGL((decompress_f32_mfma<KQ, false, true>), grid, dim3(512), 0, st, Z, ids, E, U,
                       Y, N, d, V, Zb, kz);
  else
    hipLaunchKernelGGL((decompress_f32_mfma<KQ, false, false>), grid, dim3(512), 0, st, Z, ids, E,
                       U, Y, N, d, V, Zb, kz);
  return hipGetLastError();
}

hipError_t launch_decompress_f32(int64_t N, int64_t d, int64_t k, int64_t V, const float* Z,
                                 const int32_t* ids, const float* E, const float* U, float* Y,
                                 bool gather_z, hipStream_t st, const uint16_t* Zb, int kz) {
  const int64_t blocks = (N + 127) / 128;
  const int gy = decompress_grid_split(blocks, (int)(d / kF32Chunk));
  const dim3 grid((unsigned)blocks, (unsigned)gy);
  const int dd = (int)d;
  switch (k / 16) {
    case 1: return launch_decompress_f32_kq<1>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    case 2: return launch_decompress_f32_kq<2>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    case 3: return launch_decompress_f32_kq<3>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    case 4: return launch_decompress_f32_kq<4>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    case 5: return launch_decompress_f32_kq<5>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    case 6: return launch_decompress_f32_kq<6>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    case 7: return launch_decompress_f32_kq<7>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
    default: return launch_decompress_f32_kq<8>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz);
  }
}

template <int KP, int W>
static hipError_t launch_compress_f32_kp(int64_t N, int d, int64_t V, const float* X,
                                         const int32_t* ids, const float* E, const float* U,
                                         float* Z, const float* P, hipStream_t st, uint16_t* Zb,
                                         int kz) {
  const dim3 grid((unsigned)((N + 16 * W - 1) / (16 * W)));
  if (E)
    hipLaunchKernelGGL((compress_f32_mfma<KP, true, false, W>), grid, dim3(64 * W), 0, st, X, ids, E,
                       U, Z, N, d, V, P, Zb, kz);
  else if (P)
    hipLaunchKernelGGL((compress_f32_mfma<KP, false, true, W>), grid, dim3(64 * W), 0, st, X, ids, E,
                       U, Z, N, d, V, P, Zb, kz);
  else
    hipLaunchKernelGGL((compress_f32_mfma<KP, false, false, W>), grid, dim3(64 * W), 0, st, X, ids,
                       E, U, Z, N, d, V, P, Zb, kz);
  return hipGetLastError();
}

template <int KP>
static hipError_t launch_compress_f32_w(int64_t N, int d, int64_t V, const float* X,
                                        const int32_t* ids, const float* E, const float* U, float* Z,
                                        const float* P, hipStream_t st, uint16_t* Zb, int kz) {
  // 8 waves (128 tokens) per block once those blocks fill the compute units,
  // else 4 (64 tokens)
  if ((N + 127) / 128 >= device_cu_count())
    return launch_compress_f32_kp<KP, 8>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz);
  return launch_compress_f32_kp<KP, 4>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz);
}

hipError_t launch_compress_f32(int64_t N, int64_t d, int64_t k, int64_t V, const float* X,
                               const int32_t* ids, const float* E, const float* U, float* Z,
                               const float* P, hipStream_t st, uint16_t* Zb, int kz) {
  const int dd = (int)d;
  switch (k / 16) {
    case 1: return launch_compress_f32_w<1>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 2: return launch_compress_f32_w<2>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 3: return launch_compress_f32_w<3>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 4: return launch_compress_f32_w<4>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 5: return launch_compress_f32_w<5>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 6: return launch_compress_f32_w<6>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 7: return launch_compress_f32_w<7>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
    default: return launch_compress_f32_w<8>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz);
  }
}

}  // namespace ssn

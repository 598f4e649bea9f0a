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
  return d % kF32Chunk == 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

// U rows [64 c, 64 c + 64) of U [d, ku] are one contiguous span of 64 ku
// floats (16-byte aligned with U: 256 ku bytes per chunk).  Thread tid stages
// its 16-byte pieces p = tid + T i of the span into the LDS tile of pitch
// K + 4.  SPAN false (ku == K): piece p lands whole at row 4p / K, column
// 4p % K.  SPAN (ku < K, any width): the piece's four floats go one by one
// to (row, column) = divmod(4p + e, ku); columns ku .. K - 1 are zeroed once
// by zero_pad and never written, so the tile is the zero-padded basis.
// Threads past the last piece load the last piece again (SPAN: nothing) and
// do not store it.
template <int K, int T, bool SPAN>
struct UStage {
  static constexpr int UP = K + 4;
  static constexpr int NPMAX = kF32Chunk * K / 4;
  static constexpr int FPT = (NPMAX + T - 1) / T;
  int tid, ku;
  int row0, col0, drow, dcol;   // SPAN: (row, column) of element 4 tid, and the step of 4 T elements
  __device__ __forceinline__ UStage(int tid_, int ku_) : tid(tid_), ku(SPAN ? ku_ : K) {
    if constexpr (SPAN) {
      row0 = 4 * tid / ku;
      col0 = 4 * tid - row0 * ku;
      drow = 4 * T / ku;
      dcol = 4 * T - drow * ku;
    } else {
      row0 = col0 = drow = dcol = 0;
    }
  }
  // piece tid + T i exists (threads past the last piece of the fixed-width
  // layout load the last piece again and do not store it)
  __device__ __forceinline__ bool on(int i) const {
    return SPAN ? tid + T * i < kF32Chunk * ku / 4 : (NPMAX % T == 0 || tid + T * i < NPMAX);
  }
  __device__ __forceinline__ void load(const float* __restrict__ U, int c, f32x4 (&r)[FPT]) const {
    const float* base = U + (int64_t)c * kF32Chunk * ku;
#pragma unroll
    for (int i = 0; i < FPT; ++i) {
      if constexpr (SPAN) {
        r[i] = on(i) ? *(const f32x4*)(base + 4 * (tid + T * i)) : f32x4{0.f, 0.f, 0.f, 0.f};
      } else {
        const int p = on(i) ? tid + T * i : NPMAX - 1;
        r[i] = *(const f32x4*)(base + 4 * p);
      }
    }
  }
  __device__ __forceinline__ void store(float* tile, const f32x4 (&r)[FPT]) const {
    int row = row0, col = col0;
#pragma unroll
    for (int i = 0; i < FPT; ++i) {
      if constexpr (SPAN) {
        if (on(i)) {
          int rr = row, cc = col;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            tile[rr * UP + cc] = r[i][e];
            if (++cc == ku) {
              cc = 0;
              ++rr;
            }
          }
        }
        col += dcol;
        row += drow;
        if (col >= ku) {
          col -= ku;
          ++row;
        }
      } else {
        const int p = tid + T * i;
        if (on(i)) *(f32x4*)(tile + (4 * p / K) * UP + (4 * p) % K) = r[i];
      }
    }
  }
  // columns ku .. K - 1 of the 64 rows of `tiles` consecutive tiles
  __device__ __forceinline__ void zero_pad(float* tile, int tiles) const {
    if constexpr (SPAN) {
      const int w = K - ku, n = tiles * kF32Chunk * w;
      for (int i = tid; i < n; i += T) {
        const int row = i / w;
        tile[row * UP + ku + (i - row * w)] = 0.f;
      }
    }
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
template <int KQ, bool HAS_E, bool GZ, bool SPAN>
__global__ __launch_bounds__(512) void decompress_f32_mfma(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids, const float* __restrict__ E,
    const float* __restrict__ U, float* __restrict__ Y, int64_t N, int d, int64_t V,
    const uint16_t* __restrict__ Zb, int kz, int ku) {
  static_assert(!(HAS_E && GZ), "gathered coordinates carry no additive embedding");
  constexpr int K = 16 * KQ, DC = kF32Chunk, W = 8;
  using Stage = UStage<K, 64 * W, SPAN>;
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
  const Stage stage(tid, ku);
  stage.zero_pad(&ut[0][0], 2);
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
template <int KP, bool HAS_E, bool HAS_P, int W, bool SPAN>
__global__ __launch_bounds__(64 * W) void compress_f32_mfma(
    const float* __restrict__ X, const int32_t* __restrict__ ids, const float* __restrict__ E,
    const float* __restrict__ U, float* __restrict__ Z, int64_t N, int d, int64_t V,
    const float* __restrict__ Pt, uint16_t* __restrict__ Zb, int kz, int ku) {
  static_assert(!(HAS_E && HAS_P), "the embedding is subtracted as rows or as projected rows");
  constexpr int K = 16 * KP, DC = kF32Chunk;
  using Stage = UStage<K, 64 * W, SPAN>;
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
  const Stage stage(tid, ku);
  stage.zero_pad(&ut[0][0], 2);
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
// compress / gradient projection for few tokens (the kernel above runs
// N / 64 blocks, a fraction of the chip).  Block = 16 tokens x PW waves; wave
// w walks the w-th of PW equal ranges of d with a wave-private U tile and D
// tile, so no barrier is needed until the end (a wave's LDS operations
// complete in order).  U for the next chunks travels in UD register sets;
// the MFMA loop is the one above.  The PW partial products meet in LDS and
// are added in wave order (deterministic); wave w finishes the coordinates
// KP j + h with h = w mod PW.
// ===========================================================================
template <int KP, bool HAS_E, bool HAS_P, bool SPAN, int PW, int UD>
__global__ __launch_bounds__(64 * PW) void compress_f32_split(
    const float* __restrict__ X, const int32_t* __restrict__ ids, const float* __restrict__ E,
    const float* __restrict__ U, float* __restrict__ Z, int64_t N, int d, int64_t V,
    const float* __restrict__ Pt, uint16_t* __restrict__ Zb, int kz, int ku) {
  static_assert(!(HAS_E && HAS_P), "the embedding is subtracted as rows or as projected rows");
  static_assert(UD == 1 || UD == 2, "U register sets");
  constexpr int K = 16 * KP, DC = kF32Chunk;
  using Stage = UStage<K, 64, SPAN>;
  constexpr int UP = Stage::UP, FPT = Stage::FPT;
  static_assert(KP * 64 * 4 <= DC * UP, "the partial products fit a wave's U tile");
  __shared__ __align__(16) float ut[PW][DC * UP];
  __shared__ f32x4 dt[PW][16 * 16];                // [wave][token * 16 + (cell ^ token)]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = (int64_t)blockIdx.x * 16;

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
  const Stage stage(lane, ku);
  float* const ub = ut[wave];
  stage.zero_pad(ub, 1);
  f32x4* const dw = dt[wave];
  f32x4 ust[UD][FPT];
  f32x4 xs[2][4], es[2][4];
  auto load_rows = [&](int c, f32x4(&xo)[4], f32x4(&eo)[4]) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      xo[m] = __builtin_nontemporal_load((const f32x4*)(xrow[m] + c * DC));
      if constexpr (HAS_E) eo[m] = *(const f32x4*)(erow[m] + c * DC);
    }
  };

  const int nch = d / (DC * PW), c0 = wave * nch;
  f32x4 acc[KP];
#pragma unroll
  for (int i = 0; i < KP; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // chunk i: its rows in set i % 2, its U already in the tile; chunk i + 1's
  // U in register set (i + 1) % UD
  auto body = [&](int i, auto Bc) {
    constexpr int B = decltype(Bc)::value;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int r = 4 * m + g;
      dw[r * 16 + (n16 ^ r)] = HAS_E ? xs[B][m] - es[B][m] : xs[B][m];
    }
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
    if (i + 1 < nch) {
      // the tile's reads above were issued first, so this overwrite is safe
      stage.store(ub, ust[(B + 1) % UD]);
      if (i + 1 + UD < nch) stage.load(U, c0 + i + 1 + UD, ust[(B + 1) % UD]);
      if (i + 2 < nch) load_rows(c0 + i + 2, xs[B], es[B]);
    }
  };

  stage.load(U, c0, ust[0]);
  load_rows(c0, xs[0], es[0]);
  stage.store(ub, ust[0]);
#pragma unroll
  for (int j = 1; j <= UD; ++j)
    if (j < nch) stage.load(U, c0 + j, ust[j % UD]);
  if (nch > 1) load_rows(c0 + 1, xs[1], es[1]);
  int i = 0;
  for (; i + 1 < nch; i += 2) {
    body(i, std::integral_constant<int, 0>{});
    body(i + 1, std::integral_constant<int, 1>{});
  }
  if (i < nch) body(i, std::integral_constant<int, 0>{});

  // partial products of all waves, then coordinates KP j + h (h = w mod PW)
  __syncthreads();
  f32x4* const red = (f32x4*)&ut[0][0];           // [wave][h][lane]
#pragma unroll
  for (int h = 0; h < KP; ++h) red[(wave * KP + h) * 64 + lane] = acc[h];
  __syncthreads();
#pragma unroll
  for (int h = 0; h < KP; ++h) {
    if (h % PW != wave) continue;
    f32x4 s = red[h * 64 + lane];
#pragma unroll
    for (int w2 = 1; w2 < PW; ++w2) s += red[(w2 * KP + h) * 64 + lane];
    const int col = KP * n16 + h;
    if (col >= kz) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t t = tok0 + 4 * g + r;
      if (t >= N) continue;
      float v = s[r];
      if constexpr (HAS_P) v -= Pt[clamp_id(ids[t], V) * kz + col];
      if (Zb)
        Zb[t * kz + col] = (uint16_t)f32_to_bf16(v);
      else
        Z[t * kz + col] = v;
    }
  }
}

// ===========================================================================
// Weight re-projection W <- U (U^T W) with float32 storage (the original SSN's
// step after each optimizer update, sections 4.1 and 6.1).  The columns of
// all matrices of a batch form one sequence of 16-column tiles; block b owns
// tpb consecutive tiles (a strip), one block per compute unit.  The 8 waves
// form TW = 8 / RS tile groups of RS waves: wave w = tw + TW rs owns the
// tiles tw, tw + TW, .. of the strip and row share rs.  Few tiles per block
// (small matrices) thus still keep all four SIMDs on the matrix cores.
// Pass 1, T = U^T W, over d in chunks of 32 rows: the chunk's rows of the
// strip and of U are staged into LDS row tiles (double buffered, one barrier
// per chunk, pitches chosen so that the 64 lanes of a read hit 64 banks).
// T tile (kt, j) [16 k x 16 columns] takes one MFMA per group of four rows,
// K slot g = row 4 q + g of the chunk, A = U[row][16 kt + m] and
// B = W[row][16 j + n]; wave rs takes the groups q = rs mod RS.  With RS > 1
// the RS partial sums of a tile group are added through LDS in a fixed order,
// so that every wave of the group holds the same T.  Lane (n, g) then holds
// T[16 kt + 4 g + r][16 j + n], r = 0..3: exactly its B operand of pass 2,
// where K slot g stands for coordinate 16 q + 4 g + s, so T never leaves the
// registers.  Pass 2, W = U T, in chunks of 32 RS rows, wave rs taking rows
// 32 rs .. + 31 of each: A = 16 contiguous bytes of a U row (from L2), the
// output rows parked in one of two LDS row tiles (one barrier per chunk) and
// stored by the block in 16-byte pieces (non-temporal: W is not read again).  Columns past a matrix's n (in
// its last tile) are neither used nor stored.
// ===========================================================================
struct ColumnBatchF32 {
  float* W[kMaxBatch];
  int32_t n[kMaxBatch];
  int32_t first_tile[kMaxBatch + 1];   // prefix sums of ceil(n / 16)
  int32_t count;
  int32_t tiles;                       // total tiles of the batch
  int32_t tpb;                         // tiles per block
};

constexpr int kW32Rows = 32;           // rows per pass-1 chunk
constexpr int kW32Threads = 512;
// Tiles per block at most: three per wave up to k = 80, two beyond (where
// three would spill registers).
constexpr int w32_max_tpb(int64_t k) { return k <= 80 ? 24 : 16; }

// Row pitches (floats) of tiles `width` floats wide (a multiple of 16); the
// LDS has 64 four-byte banks.  Rows 4 q + g read by lanes (n, g) at column
// 16 j + n: a pitch that is 16 mod 32 puts the four rows on four distinct
// 16-bank groups.  Rows 4 g + r written by lanes (n, g): a pitch that is 4 mod
// 16 does the same for each r.
__host__ __device__ constexpr int pitch_rows4q(int width) { return width % 32 == 0 ? width + 16 : width; }
__host__ __device__ constexpr int pitch_rows4g(int width) { return width + 4; }
constexpr int cmax3(int a, int b, int c) { return a > b ? (a > c ? a : c) : (b > c ? b : c); }

// The 16-byte piece p of a chunk of `rows` rows of the strip: row p / (4 tpb),
// tile j = (p / 4) mod tpb, columns 16 j + 4 (p mod 4) .. + 3 of the matrix
// that tile belongs to.  `on` is false past the chunk, the strip or the
// matrix's last column.
struct W32Piece {
  float* ptr;     // W + row * n + column
  int ld;         // n of the matrix
  int row;        // row within the chunk
  int lofs;       // LDS offset at pitch `pitch`
  bool on;
};
__device__ __forceinline__ W32Piece w32_piece(const ColumnBatchF32& cb, int t0, int tcount, int tpb,
                                              int p, int rows, int pitch) {
  const int row = p / (4 * tpb), q = p % (4 * tpb), j = q >> 2, sub = q & 3;
  bool on = row < rows && j < tcount;
  const int t = t0 + (on ? j : 0);
  int b = 0;
  while (b + 1 < cb.count && t >= cb.first_tile[b + 1]) ++b;
  const int col = (t - cb.first_tile[b]) * 16 + 4 * sub;
  on = on && col < cb.n[b];
  W32Piece w;
  w.ld = cb.n[b];
  w.row = on ? row : 0;
  w.ptr = cb.W[b] + (int64_t)w.row * w.ld + (on ? col : 0);
  w.lofs = on ? row * pitch + 16 * j + 4 * sub : 0;
  w.on = on;
  return w;
}

// KV: k % 4 == 0, so U rows are whole 16-byte pieces.  Otherwise a chunk of
// U (32 whole rows, one contiguous span of 32 k floats that starts 16-byte
// aligned) is read with 16-byte loads and scattered element by element into
// the zero-padded row tile, and pass 2 reads its U operands element by element.
// FG: the reparameterized layer's factor gradient (section 4.1, Eq. (3)),
// dZp = H^T GT, with H [N, din] as the single matrix of the batch, GT [N, k]
// in place of U and N rows in place of d (any N: rows past N load as zero):
// pass 1 alone, then T = GT^T H is written transposed to fg_out [din, k].
template <int KT, int CT, int RS, bool KV, bool FG>
__global__ __launch_bounds__(kW32Threads) void project_weights_f32_mfma(ColumnBatchF32 cb,
                                                                       const float* __restrict__ U,
                                                                       int d, int k, int xcd,
                                                                       float* __restrict__ fg_out) {
  static_assert(CT >= 1 && CT <= 3 && (RS == 1 || RS == 2 || RS == 4 || RS == 8), "tile groups");
  constexpr int TW = 8 / RS;                    // tile groups
  constexpr int K = 16 * KT, R1 = kW32Rows, R2 = kW32Rows * RS;
  constexpr int TMAX = TW * CT;                 // tiles per block at most
  constexpr int WP1M = 16 * TMAX + 16;          // pitch_rows4q(16 t) <= 16 t + 16
  constexpr int WP2M = 16 * TMAX + 4;           // pitch_rows4g(16 t)
  constexpr int UP1 = pitch_rows4q(K);
  constexpr int NP1 = (R1 * 4 * TMAX + kW32Threads - 1) / kW32Threads;
  constexpr int NP2 = (R2 * 4 * TMAX + kW32Threads - 1) / kW32Threads;
  constexpr int NUP = (R1 * K / 4 + kW32Threads - 1) / kW32Threads;   // U pieces per thread
  constexpr int QN = 8 / RS;                    // row groups per chunk and wave (pass 1)
  // pass 1: two W and two U row tiles; reduction: 8 waves' partial T; pass 2:
  // two output row tiles
  constexpr int S1 = 2 * R1 * WP1M + 2 * R1 * UP1;
  constexpr int SR = RS > 1 ? 8 * KT * CT * 256 : 0;
  constexpr int S2 = 2 * R2 * WP2M;
  __shared__ __align__(16) float smem[cmax3(S1, SR, S2)];
  float* const wtile = smem;                    // buffer b at b * R1 * WP1M
  float* const utile = smem + 2 * R1 * WP1M;    // buffer b at b * R1 * UP1

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int tw = wave % TW, rs = wave / TW;
  const int tpb = cb.tpb;
  const int WP1 = pitch_rows4q(16 * tpb);
  const int WP2 = pitch_rows4g(16 * tpb);
  // XCD order: neighbouring strips, which share the 128-byte lines at their
  // boundary, run on the same XCD (blocks go to the 8 XCDs round robin)
  const int bx = xcd ? (int)((blockIdx.x % 8u) * (gridDim.x / 8u) + blockIdx.x / 8u) : (int)blockIdx.x;
  const int t0 = bx * tpb;
  const int tcount = min(tpb, cb.tiles - t0);
  const int nch1 = FG ? (d + R1 - 1) / R1 : d / R1, nch2 = (d + R2 - 1) / R2;
  // this wave's tiles: tw + TW v for v < nv
  const int nv = tcount > tw ? min(CT, (tcount - tw + TW - 1) / TW) : 0;

  W32Piece wp[NP1];
#pragma unroll
  for (int i = 0; i < NP1; ++i) wp[i] = w32_piece(cb, t0, tcount, tpb, tid + kW32Threads * i, R1, WP1);
  int uo[NUP], us[NUP];
  bool uon[NUP];
#pragma unroll
  for (int i = 0; i < NUP; ++i) {
    const int p = tid + kW32Threads * i;
    if constexpr (KV) {
      const int row = p / (k / 4), cg = p % (k / 4);
      uon[i] = row < R1;
      us[i] = uon[i] ? row * k + 4 * cg : 0;
      uo[i] = uon[i] ? row * UP1 + 4 * cg : 0;
    } else {
      // floats 4 p .. 4 p + 3 of the chunk's span
      uon[i] = p < R1 * k / 4;
      us[i] = uon[i] ? 4 * p : 0;
      uo[i] = 0;
    }
  }
  // columns k .. K - 1 of the U tiles stay zero
  for (int i = tid; i < 2 * R1 * UP1; i += kW32Threads) utile[i] = 0.f;

  f32x4 wv[NP1], uv[NUP];
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int i = 0; i < NP1; ++i) {
      const f32x4* src = (const f32x4*)(wp[i].ptr + (int64_t)c * R1 * wp[i].ld);
      const bool ok = wp[i].on && (!FG || c * R1 + wp[i].row < d);
      if constexpr (RS == 1)
        wv[i] = ok ? __builtin_nontemporal_load(src) : f32x4{0.f, 0.f, 0.f, 0.f};
      else
        wv[i] = ok ? *src : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < NUP; ++i) {
      const int64_t e0 = (int64_t)c * R1 * k + us[i];
      if constexpr (FG) {
        // elements past the N k floats of GT load as zero
        const int64_t lim = (int64_t)d * k;
        if (uon[i] && e0 + 4 <= lim) {
          uv[i] = *(const f32x4*)(U + e0);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) uv[i][e] = (uon[i] && e0 + e < lim) ? U[e0 + e] : 0.f;
        }
      } else {
        uv[i] = uon[i] ? *(const f32x4*)(U + e0) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  };
  auto store_chunk = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NP1; ++i)
      if (wp[i].on) *(f32x4*)(wtile + buf * R1 * WP1M + wp[i].lofs) = wv[i];
#pragma unroll
    for (int i = 0; i < NUP; ++i)
      if (uon[i]) {
        if constexpr (KV) {
          *(f32x4*)(utile + buf * R1 * UP1 + uo[i]) = uv[i];
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int idx = us[i] + e, row = idx / k;
            utile[buf * R1 * UP1 + row * UP1 + (idx - row * k)] = uv[i][e];
          }
        }
      }
  };

  // A operand of pass 2: U[rb + 16 dt + n16][16 q + 4 g .. + 3] for chunk c,
  // rb = 32 RS c + 32 rs (zero past k; d is a multiple of 32, so rb < d
  // keeps all 32 rows in range)
  auto load_ua = [&](int c, f32x4(&v)[2][KT]) {
    const int rb = c * R2 + 32 * rs;
#pragma unroll
    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
      for (int q = 0; q < KT; ++q) {
        const int col = 16 * q + 4 * g;
        const float* src = U + (int64_t)(rb < d ? rb + 16 * dt + n16 : 0) * k + col;
        if constexpr (KV) {
          v[dt][q] = (rb < d && col < k) ? *(const f32x4*)src : f32x4{0.f, 0.f, 0.f, 0.f};
        } else {
#pragma unroll
          for (int s = 0; s < 4; ++s) v[dt][q][s] = (rb < d && col + s < k) ? src[s] : 0.f;
        }
      }
  };

  // The whole computation for a wave that owns NV tiles (NV known at compile
  // time, so that neither pass branches between its MFMAs).  Every wave runs
  // the same barriers and its share of the block's loads and stores.
  auto run = [&](auto NVc) {
    constexpr int NV = decltype(NVc)::value;
    constexpr int NA = NV > 0 ? NV : 1;
    constexpr int PD = KT * NA <= 4 ? 2 : 1;    // pass-2 U operand sets in flight

    // ---- pass 1: T = U^T W ----
    f32x4 acc[KT][NA];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int v = 0; v < NA; ++v) acc[kt][v] = f32x4{0.f, 0.f, 0.f, 0.f};
    load_chunk(0);
    __syncthreads();                            // the zeroed U tiles
    store_chunk(0);
    if (nch1 > 1) load_chunk(1);
    for (int c = 0; c < nch1; ++c) {
      __syncthreads();                          // chunk c in buffer c % 2; chunk c - 1 fully read
      if (c + 1 < nch1) {
        store_chunk((c + 1) & 1);
        if (c + 2 < nch1) load_chunk(c + 2);
      }
      if constexpr (NV > 0) {
        const float* ub = utile + (c & 1) * R1 * UP1;
        const float* wb = wtile + (c & 1) * R1 * WP1M;
#pragma unroll
        for (int qi = 0; qi < QN; ++qi) {
          const int row = 4 * (rs + RS * qi) + g;
          float a[KT], b[NV];
#pragma unroll
          for (int kt = 0; kt < KT; ++kt) a[kt] = ub[row * UP1 + 16 * kt + n16];
#pragma unroll
          for (int v = 0; v < NV; ++v) b[v] = wb[row * WP1 + 16 * (tw + TW * v) + n16];
#pragma unroll
          for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) acc[kt][v] = mfma16x16x4f32(a[kt], b[v], acc[kt][v]);
        }
      }
    }
    __syncthreads();                            // pass 1 done with the row tiles

    if constexpr (RS > 1) {
      // partial T of wave w at red[(w KT CT + e) 64 + lane], element
      // e = kt CT + v.  Wave rs of a group adds the partials of elements
      // e = rs mod RS in the order of the group's waves and stores the total
      // over the first partial; every wave then reads its T back.  (The waves
      // of a group own the same tiles, so they agree on NV.)
      constexpr int E = KT * CT, NE = (E + RS - 1) / RS;
      f32x4* const red = (f32x4*)smem;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int v = 0; v < NV; ++v) red[(wave * E + kt * CT + v) * 64 + lane] = acc[kt][v];
      __syncthreads();
      f32x4 tot[NE];
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const int e = rs + RS * i;
        if (e < E && e % CT < NV) {
          f32x4 s = red[(tw * E + e) * 64 + lane];
#pragma unroll
          for (int r2 = 1; r2 < RS; ++r2) s += red[((tw + TW * r2) * E + e) * 64 + lane];
          tot[i] = s;
        }
      }
      __syncthreads();                          // every partial read
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const int e = rs + RS * i;
        if (e < E && e % CT < NV) red[(tw * E + e) * 64 + lane] = tot[i];
      }
      __syncthreads();
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int v = 0; v < NV; ++v) acc[kt][v] = red[(tw * E + kt * CT + v) * 64 + lane];
      __syncthreads();                          // totals read before pass 2 parks rows
    }

    if constexpr (FG) {
      // lane (n16, g) holds T[16 kt + 4 g + r][16 j + n16]: dZp row 16 j + n16
      // (of din), columns 16 kt + 4 g + r (of k); one wave per tile group writes
      if (rs == 0) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int col = 16 * (t0 + tw + TW * v) + n16;
          if (col >= cb.n[0]) continue;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt) {
            const int kc = 16 * kt + 4 * g;
            float* dst = fg_out + (int64_t)col * k + kc;
            if (KV && kc < k && (((uintptr_t)fg_out & 15u) == 0)) {
              *(f32x4*)dst = acc[kt][v];
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (kc + r < k) dst[r] = acc[kt][v][r];
            }
          }
        }
      }
      return;
    }

    // ---- pass 2: W = U T ----
    W32Piece op[NP2];
#pragma unroll
    for (int i = 0; i < NP2; ++i) op[i] = w32_piece(cb, t0, tcount, tpb, tid + kW32Threads * i, R2, WP2);
    f32x4 ua[PD][2][KT];
    // chunk c parks its rows in output tile c % 2: the barrier after chunk
    // c + 1 is parked orders the stores of chunk c before chunk c + 2 parks
    auto body2 = [&](int c, auto Sc) {
      constexpr int S = decltype(Sc)::value;
      float* const ot = smem + (c & 1) * R2 * WP2M;
      if constexpr (NV > 0) {
        if constexpr (PD == 2) {
          if (c + 1 < nch2) load_ua(c + 1, ua[S ^ 1]);
        }
        const int rbase = 32 * rs;
        if (c * R2 + rbase < d) {
          // the 2 NV output tiles take their MFMAs in turn, so that no MFMA
          // waits for the result of the one before
          f32x4 o[2][NV];
#pragma unroll
          for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int v = 0; v < NV; ++v) o[dt][v] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int q = 0; q < KT; ++q)
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
              for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int v = 0; v < NV; ++v)
                  o[dt][v] = mfma16x16x4f32(ua[S][dt][q][s], acc[q][v][s], o[dt][v]);
          // lane (n16, g): rows rbase + 16 dt + 4 g + r, column 16 j + n16
#pragma unroll
          for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int v = 0; v < NV; ++v)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                ot[(rbase + 16 * dt + 4 * g + r) * WP2 + 16 * (tw + TW * v) + n16] = o[dt][v][r];
        }
        if constexpr (PD == 1) {
          if (c + 1 < nch2) load_ua(c + 1, ua[0]);
        }
      }
      __syncthreads();                          // the chunk's output rows are parked
#pragma unroll
      for (int i = 0; i < NP2; ++i)
        if (op[i].on && c * R2 + op[i].row < d)
          __builtin_nontemporal_store(*(const f32x4*)(ot + op[i].lofs),
                                      (f32x4*)(op[i].ptr + (int64_t)c * R2 * op[i].ld));
    };
    if constexpr (NV > 0) load_ua(0, ua[0]);
    int c = 0;
    if constexpr (PD == 2) {
      for (; c + 1 < nch2; c += 2) {
        body2(c, std::integral_constant<int, 0>{});
        body2(c + 1, std::integral_constant<int, 1>{});
      }
    }
    for (; c < nch2; ++c) body2(c, std::integral_constant<int, 0>{});
  };
  if (nv >= 3) {
    if constexpr (CT >= 3) run(std::integral_constant<int, 3>{});
  } else if (nv == 2) {
    if constexpr (CT >= 2) run(std::integral_constant<int, 2>{});
  } else if (nv == 1) {
    run(std::integral_constant<int, 1>{});
  } else {
    run(std::integral_constant<int, 0>{});
  }
}

// ===========================================================================
// Launchers.
// ===========================================================================
template <int KQ, bool SPAN>
static hipError_t launch_decompress_f32_kq(dim3 grid, int64_t N, int d, int64_t V, const float* Z,
                                           const int32_t* ids, const float* E, const float* U,
                                           float* Y, bool gather_z, hipStream_t st,
                                           const uint16_t* Zb, int kz, int ku) {
  if (E)
    hipLaunchKernelGGL((decompress_f32_mfma<KQ, true, false, SPAN>), grid, dim3(512), 0, st, Z, ids, E,
                       U, Y, N, d, V, Zb, kz, ku);
  else if (gather_z)
    hipLaunchKernelGGL((decompress_f32_mfma<KQ, false, true, SPAN>), grid, dim3(512), 0, st, Z, ids, E,
                       U, Y, N, d, V, Zb, kz, ku);
  else
    hipLaunchKernelGGL((decompress_f32_mfma<KQ, false, false, SPAN>), grid, dim3(512), 0, st, Z, ids,
                       E, U, Y, N, d, V, Zb, kz, ku);
  return hipGetLastError();
}

template <int KQ>
static hipError_t launch_decompress_f32_span(dim3 grid, int64_t N, int d, int64_t V, const float* Z,
                                             const int32_t* ids, const float* E, const float* U,
                                             float* Y, bool gather_z, hipStream_t st,
                                             const uint16_t* Zb, int kz, int ku) {
  return ku == 16 * KQ
             ? launch_decompress_f32_kq<KQ, false>(grid, N, d, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku)
             : launch_decompress_f32_kq<KQ, true>(grid, N, d, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
}

hipError_t launch_decompress_f32(int64_t N, int64_t d, int64_t k, int64_t V, const float* Z,
                                 const int32_t* ids, const float* E, const float* U, float* Y,
                                 bool gather_z, hipStream_t st, const uint16_t* Zb, int kz) {
  const int64_t blocks = (N + 127) / 128;
  const int gy = decompress_grid_split(blocks, (int)(d / kF32Chunk));
  const dim3 grid((unsigned)blocks, (unsigned)gy);
  const int dd = (int)d, ku = (int)k;
  switch ((k + 15) / 16) {
    case 1: return launch_decompress_f32_span<1>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    case 2: return launch_decompress_f32_span<2>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    case 3: return launch_decompress_f32_span<3>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    case 4: return launch_decompress_f32_span<4>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    case 5: return launch_decompress_f32_span<5>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    case 6: return launch_decompress_f32_span<6>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    case 7: return launch_decompress_f32_span<7>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
    default: return launch_decompress_f32_span<8>(grid, N, dd, V, Z, ids, E, U, Y, gather_z, st, Zb, kz, ku);
  }
}

template <int KP, int W, bool SPAN>
static hipError_t launch_compress_f32_kp(int64_t N, int d, int64_t V, const float* X,
                                         const int32_t* ids, const float* E, const float* U,
                                         float* Z, const float* P, hipStream_t st, uint16_t* Zb,
                                         int kz, int ku) {
  const dim3 grid((unsigned)((N + 16 * W - 1) / (16 * W)));
  if (E)
    hipLaunchKernelGGL((compress_f32_mfma<KP, true, false, W, SPAN>), grid, dim3(64 * W), 0, st, X, ids,
                       E, U, Z, N, d, V, P, Zb, kz, ku);
  else if (P)
    hipLaunchKernelGGL((compress_f32_mfma<KP, false, true, W, SPAN>), grid, dim3(64 * W), 0, st, X, ids,
                       E, U, Z, N, d, V, P, Zb, kz, ku);
  else
    hipLaunchKernelGGL((compress_f32_mfma<KP, false, false, W, SPAN>), grid, dim3(64 * W), 0, st, X,
                       ids, E, U, Z, N, d, V, P, Zb, kz, ku);
  return hipGetLastError();
}

template <int KP, bool SPAN>
static hipError_t launch_compress_f32_split(int64_t N, int d, int64_t V, const float* X,
                                            const int32_t* ids, const float* E, const float* U,
                                            float* Z, const float* P, hipStream_t st, uint16_t* Zb,
                                            int kz, int ku) {
  constexpr int PW = 4, UD = KP <= 4 ? 2 : 1;
  const dim3 grid((unsigned)((N + 15) / 16));
  if (E)
    hipLaunchKernelGGL((compress_f32_split<KP, true, false, SPAN, PW, UD>), grid, dim3(64 * PW), 0, st, X,
                       ids, E, U, Z, N, d, V, P, Zb, kz, ku);
  else if (P)
    hipLaunchKernelGGL((compress_f32_split<KP, false, true, SPAN, PW, UD>), grid, dim3(64 * PW), 0, st, X,
                       ids, E, U, Z, N, d, V, P, Zb, kz, ku);
  else
    hipLaunchKernelGGL((compress_f32_split<KP, false, false, SPAN, PW, UD>), grid, dim3(64 * PW), 0, st,
                       X, ids, E, U, Z, N, d, V, P, Zb, kz, ku);
  return hipGetLastError();
}

template <int KP>
static hipError_t launch_compress_f32_w(int64_t N, int d, int64_t V, const float* X,
                                        const int32_t* ids, const float* E, const float* U, float* Z,
                                        const float* P, hipStream_t st, uint16_t* Zb, int kz, int ku) {
  // 8 waves (128 tokens) per block once those blocks fill the compute units,
  // else 4 (64 tokens); U rows of any width other than 16 KP are staged
  // span-wise.  With at most half as many 64-token blocks as compute units,
  // d is split over the 4 waves of 16-token blocks instead (measured on
  // MI355X, compress / projection: N = 2048, d = 2048, k = 40: 53 -> 22 us;
  // N = 4096, d = 5120, k = 51: 152 -> 62 us; N = 8192, d = 2048: 57 ->
  // 43 us; but N = 12288, d = 5120: 167 us against 185 us split).
  const int64_t cus = device_cu_count();
  const bool eight = (N + 127) / 128 >= cus, span = ku != 16 * KP;
  if (2 * ((N + 63) / 64) <= cus && d % (4 * kF32Chunk) == 0)
    return span ? launch_compress_f32_split<KP, true>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz, ku)
                : launch_compress_f32_split<KP, false>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
  if (eight && !span) return launch_compress_f32_kp<KP, 8, false>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
  if (eight) return launch_compress_f32_kp<KP, 8, true>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
  if (!span) return launch_compress_f32_kp<KP, 4, false>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
  return launch_compress_f32_kp<KP, 4, true>(N, d, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
}

hipError_t launch_compress_f32(int64_t N, int64_t d, int64_t k, int64_t V, const float* X,
                               const int32_t* ids, const float* E, const float* U, float* Z,
                               const float* P, hipStream_t st, uint16_t* Zb, int kz) {
  const int dd = (int)d, ku = (int)k;
  switch ((k + 15) / 16) {
    case 1: return launch_compress_f32_w<1>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    case 2: return launch_compress_f32_w<2>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    case 3: return launch_compress_f32_w<3>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    case 4: return launch_compress_f32_w<4>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    case 5: return launch_compress_f32_w<5>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    case 6: return launch_compress_f32_w<6>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    case 7: return launch_compress_f32_w<7>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
    default: return launch_compress_f32_w<8>(N, dd, V, X, ids, E, U, Z, P, st, Zb, kz, ku);
  }
}

template <int KT, int CT, int RS, bool FG>
static hipError_t launch_weights_f32_cfg(const ColumnBatchF32& cb, const float* U, int d, int k,
                                         float* fg_out, hipStream_t st) {
  const unsigned grid = (unsigned)((cb.tiles + cb.tpb - 1) / cb.tpb);
  const int xcd = grid % 8 == 0 ? 1 : 0;
  if (k % 4 == 0)
    hipLaunchKernelGGL((project_weights_f32_mfma<KT, CT, RS, true, FG>), dim3(grid), dim3(kW32Threads), 0,
                       st, cb, U, d, k, xcd, fg_out);
  else
    hipLaunchKernelGGL((project_weights_f32_mfma<KT, CT, RS, false, FG>), dim3(grid), dim3(kW32Threads), 0,
                       st, cb, U, d, k, xcd, fg_out);
  return hipGetLastError();
}

// Tile groups by tiles per block: 8 groups of one wave for tpb >= 8 (CT =
// ceil(tpb / 8) tiles per wave), 4 groups of 2 waves for 4..7, 2 of 4 for 2..3,
// one of 8 for a single tile.
template <int KT, bool FG>
static hipError_t launch_weights_f32_kt(const ColumnBatchF32& cb, const float* U, int d, int k,
                                        float* fg_out, hipStream_t st) {
  const int tpb = cb.tpb;
  if constexpr (KT <= 5) {
    if (tpb >= 17) return launch_weights_f32_cfg<KT, 3, 1, FG>(cb, U, d, k, fg_out, st);
  }
  if (tpb >= 9) return launch_weights_f32_cfg<KT, 2, 1, FG>(cb, U, d, k, fg_out, st);
  if (tpb == 8) return launch_weights_f32_cfg<KT, 1, 1, FG>(cb, U, d, k, fg_out, st);
  if (tpb >= 5) return launch_weights_f32_cfg<KT, 2, 2, FG>(cb, U, d, k, fg_out, st);
  if (tpb == 4) return launch_weights_f32_cfg<KT, 1, 2, FG>(cb, U, d, k, fg_out, st);
  if (tpb == 3) return launch_weights_f32_cfg<KT, 2, 4, FG>(cb, U, d, k, fg_out, st);
  if (tpb == 2) return launch_weights_f32_cfg<KT, 1, 4, FG>(cb, U, d, k, fg_out, st);
  return launch_weights_f32_cfg<KT, 1, 8, FG>(cb, U, d, k, fg_out, st);
}

template <bool FG>
static hipError_t launch_strips_f32(ColumnBatchF32& cb, const float* U, int d, int k, float* fg_out,
                                    hipStream_t st) {
  // one block per compute unit while a strip fits the LDS tiles
  const int cus = device_cu_count();
  const int tpb = (cb.tiles + cus - 1) / cus, tmax = w32_max_tpb(k);
  cb.tpb = tpb < 1 ? 1 : (tpb > tmax ? tmax : tpb);
  switch ((k + 15) / 16) {
    case 1: return launch_weights_f32_kt<1, FG>(cb, U, d, k, fg_out, st);
    case 2: return launch_weights_f32_kt<2, FG>(cb, U, d, k, fg_out, st);
    case 3: return launch_weights_f32_kt<3, FG>(cb, U, d, k, fg_out, st);
    case 4: return launch_weights_f32_kt<4, FG>(cb, U, d, k, fg_out, st);
    case 5: return launch_weights_f32_kt<5, FG>(cb, U, d, k, fg_out, st);
    case 6: return launch_weights_f32_kt<6, FG>(cb, U, d, k, fg_out, st);
    case 7: return launch_weights_f32_kt<7, FG>(cb, U, d, k, fg_out, st);
    default: return launch_weights_f32_kt<8, FG>(cb, U, d, k, fg_out, st);
  }
}

bool weights_f32_uses_mfma(int64_t d, int64_t k) {
  return d % kW32Rows == 0 && d > 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

hipError_t launch_project_weights_f32(int count, int64_t d, const int64_t* n, int64_t k,
                                      float* const* W, const float* U, hipStream_t st) {
  ColumnBatchF32 cb{};
  int nb = 0;
  int32_t acc = 0;
  for (int b = 0; b < count; ++b) {
    if (n[b] == 0) continue;
    cb.W[nb] = W[b];
    cb.n[nb] = (int32_t)n[b];
    cb.first_tile[nb] = acc;
    acc += (int32_t)((n[b] + 15) / 16);
    ++nb;
  }
  if (nb == 0) return hipSuccess;
  for (int b = nb; b <= kMaxBatch; ++b) cb.first_tile[b] = acc;
  cb.count = nb;
  cb.tiles = acc;
  return launch_strips_f32<false>(cb, U, (int)d, (int)k, nullptr, st);
}

bool factor_grad_f32_uses_mfma(int64_t N, int64_t din, int64_t k) {
  return N >= 0 && N <= INT32_MAX && din >= 1 && din % 4 == 0 && din <= INT32_MAX / 2 && k >= 1 &&
         k <= 128;
}

hipError_t launch_factor_grad_f32(int64_t N, int64_t din, int64_t k, const float* H, const float* GT,
                                  float* dZp, hipStream_t st) {
  ColumnBatchF32 cb{};
  cb.W[0] = const_cast<float*>(H);    // read only: the factor-gradient mode has no second pass
  cb.n[0] = (int32_t)din;
  const int32_t tiles = (int32_t)((din + 15) / 16);
  cb.first_tile[0] = 0;
  for (int b = 1; b <= kMaxBatch; ++b) cb.first_tile[b] = tiles;
  cb.count = 1;
  cb.tiles = tiles;
  return launch_strips_f32<true>(cb, GT, (int)N, (int)k, dZp, st);
}

}  // namespace ssn

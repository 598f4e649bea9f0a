// Stage-boundary codec with float32 storage on the matrix cores:
// v_mfma_f32_16x16x4_f32 multiplies float32 operands and accumulates in
// float32, so no operand is split.  Paper: section 4.1, Eq. (2) --
// Z = (X - E[ids]) U, X' = E[ids] + Z U^T; the gradient forms are the same
// kernels without the embedding.
//
// The kernels walk d in 64-wide chunks (256 contiguous bytes of a float32
// row) and stage the chunk's 64 rows of U [d, ku] (any ku <= 128) into a
// row-major LDS tile K = 16 ceil(ku / 16) wide (pitch K + 4 floats, zero past
// ku): the many-token kernels once per block, double buffered, one barrier
// per chunk, their activation and embedding rows moving as 4 rows x 256
// contiguous bytes per instruction; the few-token compress / projection once
// per wave, with no barrier.
#include "ssn_device.h"
#include "ssn_launch.h"

#include <type_traits>

namespace ssn {

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
  // HAS_P: table row offsets of the epilogue's tokens 4 g + r, looked up now
  int64_t prow[HAS_P ? 4 : 1];
  if constexpr (HAS_P) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t t = tok0 + 4 * g + r;
      prow[r] = t < N ? clamp_id(ids[t], V) * kz : 0;
    }
  }

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
      if constexpr (HAS_P) v -= Pt[prow[r] + col];
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
// w walks the w-th of PW equal ranges of d with a wave-private U tile and
// its A operands read straight from the rows, so no barrier is needed until
// the end (a wave's LDS operations complete in order).  U for the next chunks travels in UD register sets;
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

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = (int64_t)blockIdx.x * 16;
  // HAS_P: table row offsets of the epilogue's tokens 4 g + r, looked up now
  int64_t prow[HAS_P ? 4 : 1];
  if constexpr (HAS_P) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t t = tok0 + 4 * g + r;
      prow[r] = t < N ? clamp_id(ids[t], V) * kz : 0;
    }
  }

  // A operand straight from the rows: lane (n16, g) reads d = 16 q + 4 g ..
  // + 3 of token n16 (16 tokens x 64 contiguous bytes per instruction) and
  // forms X - E in registers
  int64_t tn = tok0 + n16;
  tn = tn < N ? tn : N - 1;
  const float* const xa = X + tn * d + 4 * g;
  const float* const ea = HAS_E ? E + clamp_id(ids[tn], V) * d + 4 * g : nullptr;
  const Stage stage(lane, ku);
  float* const ub = ut[wave];
  stage.zero_pad(ub, 1);
  f32x4 ust[UD][FPT];
  f32x4 xs[2][4], es[2][4];
  auto load_rows = [&](int c, f32x4(&xo)[4], f32x4(&eo)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      xo[q] = __builtin_nontemporal_load((const f32x4*)(xa + c * DC + 16 * q));
      if constexpr (HAS_E) eo[q] = *(const f32x4*)(ea + c * DC + 16 * q);
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
    for (int q = 0; q < 4; ++q) {
      const f32x4 a = HAS_E ? xs[B][q] - es[B][q] : xs[B][q];
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
      if constexpr (HAS_P) v -= Pt[prow[r] + col];
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
  constexpr int PW = KP <= 4 ? 8 : 4, UD = KP <= 2 ? 2 : 1;
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
  // span-wise.  With at most three quarters as many 64-token blocks as
  // compute units, d is split over the waves of 16-token blocks instead
  // (measured on MI355X, compress / projection: N = 2048, d = 2048, k = 40:
  // 53 / 53 -> 21 / 17 us; N = 4096, d = 5120, k = 51: 152 / 150 -> 54 /
  // 45 us; N = 8192, d = 2048: 57 / 56 -> 40 / 35 us; N = 12288, d = 5120:
  // 167 / 182 -> 164 / 146 us; but N = 16384, d = 4096, k = 64: 130 / 108
  // us on the 64-token blocks against 166 / 143 us split).
  const int64_t cus = device_cu_count();
  const bool eight = (N + 127) / 128 >= cus, span = ku != 16 * KP;
  if (4 * ((N + 63) / 64) <= 3 * cus && d % ((KP <= 4 ? 8 : 4) * kF32Chunk) == 0)
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

}  // namespace ssn

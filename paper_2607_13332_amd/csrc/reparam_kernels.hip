// Reparameterized-SSN factor gradient (section 4.1, Eq. (3)).
//
// An output projection W [din, d] is stored as its factor Zp [din, k] with
// W = Zp U^T; the optimizer needs dL/dZp = (dL/dW) U = H^T (G U).  The
// gradient projection GT = G U [N, k] is formed by the codec's projection
// kernel; this file contracts it with the layer input H [N, din] over the
// tokens:
//     dZp[i, c] = sum_t H[t, i] GT[t, c]            (float32 result)
#include "ssn_device.h"
#include "ssn_launch.h"

#include <type_traits>

namespace ssn {

constexpr int kFgRows = 32;      // tokens per chunk (one K step)
// 16-column tiles of din per block: 32 (512 columns) for k <= 64; 16 for
// k > 64, whose accumulators for 32 tiles would not fit in the registers of
// two waves per SIMD (they spilled)
constexpr int fg_tiles(int kt) { return kt > 4 ? 16 : 32; }
constexpr int kFgThreads = 512;  // 8 waves, four tiles each
constexpr int kFgTargetBlocks = 256;
constexpr int kFgDepth = 2;      // chunks in flight in registers (3 measured slower)
// 16-column tiles per block of the fused backward pass for k <= 64.  16-tile
// blocks (two per compute unit, fewer token splits) measured slower on
// MI355X: backward at N = 32768, din = 14336, k = 64 451 -> 492 us.
constexpr int kFusedTiles = 32;

// ===========================================================================
// MFMA kernel, bf16 H.  Block (column block x, token split y) owns din
// columns [16 TILES x, 16 TILES (x + 1)) (512 columns for k <= 64) and
// tokens [y*tps, (y+1)*tps).  Per chunk of 32 tokens the block loads H rows
// (16-byte pieces, 2 TILES per row) into a row-major LDS tile, and GT rows split into
// bf16 hi + lo parts into two row-major LDS tiles (zero past k).  Both MFMA
// operands are token-contiguous fragments read with LDS transpose reads:
// A = H^T (16 din x 32 tokens), B = GT (32 tokens x 16 of k), two MFMAs per
// pair (hi, lo) so GT keeps ~fp32 accuracy.  Wave w owns tiles w + 8j for
// all of k.  The wide column block makes each block's GT rows serve 512
// columns (GT comes from L2 once per block).  The block writes its
// partial sums for its token split; a second kernel adds the splits in order
// (deterministic).
// ===========================================================================
// FULL: every block owns TILES whole tiles, every split a whole number of
// chunks and every GT chunk is whole 16-byte pieces for all threads (k a
// multiple of 64).  Then every load is issued unconditionally (the prefetch
// past the last chunk re-reads the last chunk): with conditional loads the
// wait before parking a chunk compiles to a full drain of the prefetch.
// NTH: H is read with non-temporal loads (each element is read once).
template <int KT, bool K4, bool FULL = false, bool NTH = false>
__global__ __launch_bounds__(kFgThreads) void factor_grad_bf16(const uint16_t* __restrict__ H,
                                                               const float* __restrict__ GT,
                                                               float* __restrict__ out, int64_t N,
                                                               int din, int k, int64_t tps) {
  constexpr int R = kFgRows, NT = kFgThreads, NW = NT / kWave;
  constexpr int TILES = fg_tiles(KT);
  constexpr int CT = TILES / NW;                       // tiles per wave
  constexpr int HP = 2 * TILES, WP = HP + 1;           // H pieces per row, pitch in pieces
  constexpr int RP = NT / HP;                          // H rows per pass
  constexpr int KS2 = (KT + 1) / 2, KW = 32 * KS2;   // GT tile width (bf16)
  constexpr int GPI = KW + 8;                          // GT tile pitch (bf16)
  constexpr int NHP = R / RP;                          // H pieces per thread per chunk
  static_assert(NT % HP == 0 && R % RP == 0 && R % 32 == 0, "piece mapping");
  constexpr int NGQ = K4 ? (R * KW / 4 + NT - 1) / NT : (R * KW + NT - 1) / NT;
  __shared__ u32x4 ht[2][R * WP];
  __shared__ __align__(16) uint16_t gtl[2][2][R * GPI];   // [buffer][hi / lo][row * GPI + col]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = lane & 15, g = lane >> 4;
  const int col0 = (int)blockIdx.x * 16 * TILES;
  const int tcount = min(TILES, din / 16 - (int)blockIdx.x * TILES);
  const int64_t t_begin = (int64_t)blockIdx.y * tps;
  const int64_t t_end = min(N, t_begin + tps);
  const int nch = (int)((t_end - t_begin + R - 1) / R);

  // GT padding columns k .. KW are never written below
  for (int i = tid; i < 2 * 2 * R * GPI / 8; i += NT) ((u32x4*)&gtl[0][0][0])[i] = u32x4{0u, 0u, 0u, 0u};

  const int h = tid % HP, row0 = tid / HP;          // row0 < RP
  const bool hok = h < 2 * tcount;
  const uint16_t* hsrc = H + (t_begin + row0) * din + col0 + 8 * h;

  // D register sets: chunk c travels in set c % D (two when k > 64, where
  // three sets would not fit in registers)
  constexpr int D = KT > 4 ? 2 : kFgDepth;
  u32x4 hv[D][NHP];
  float gv[D][NGQ][K4 ? 4 : 1];
  auto load = [&](int c, u32x4 (&hr)[NHP], float (&gr)[NGQ][K4 ? 4 : 1]) __attribute__((always_inline)) {
    const int64_t r0 = (int64_t)c * R;
#pragma unroll
    for (int i = 0; i < NHP; ++i) {
      const int64_t t = t_begin + r0 + row0 + RP * i;
      if constexpr (FULL)
        hr[i] = ldg<NTH>(hsrc + (r0 + RP * i) * din);
      else
        hr[i] = (hok && t < t_end) ? ldg<NTH>(hsrc + (r0 + RP * i) * din) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < NGQ; ++j) {
      const int q = tid + NT * j;
      if constexpr (FULL) {
        // threads past the chunk's R * k / 4 pieces (k = 32: half of them)
        // load its last piece again; the park below skips them
        const int qq = q < R * (k / 4) ? q : R * (k / 4) - 1;
        const int row = qq / (k / 4), c4 = qq - (qq / (k / 4)) * (k / 4);
        const f32x4 v = *(const f32x4*)(GT + (t_begin + r0 + row) * k + 4 * c4);
        gr[j][0] = v[0]; gr[j][1] = v[1]; gr[j][2] = v[2]; gr[j][3] = v[3];
      } else if constexpr (K4) {
        const int row = q / (k / 4), c4 = q - (q / (k / 4)) * (k / 4);
        const int64_t t = t_begin + r0 + row;
        const bool ok = q < R * (k / 4) && t < t_end;
        const f32x4 v = ok ? *(const f32x4*)(GT + t * k + 4 * c4) : f32x4{0.f, 0.f, 0.f, 0.f};
        gr[j][0] = v[0]; gr[j][1] = v[1]; gr[j][2] = v[2]; gr[j][3] = v[3];
      } else {
        const int row = q / k;
        const int64_t t = t_begin + r0 + row;
        gr[j][0] = (q < R * k && t < t_end) ? GT[t * k + (q - row * k)] : 0.f;
      }
    }
  };
  auto park = [&](int buf, const u32x4 (&hr)[NHP], const float (&gr)[NGQ][K4 ? 4 : 1]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NHP; ++i) ht[buf][(row0 + RP * i) * WP + h] = hr[i];
#pragma unroll
    for (int j = 0; j < NGQ; ++j) {
      const int q = tid + NT * j;
      if constexpr (K4) {
        if (q < R * (k / 4)) {
          const int row = q / (k / 4), c4 = q - (q / (k / 4)) * (k / 4);
          uint32_t hi[2], lo[2];
#pragma unroll
          for (int m = 0; m < 2; ++m) {
            const uint32_t h0 = f32_to_bf16(gr[j][2 * m]), h1 = f32_to_bf16(gr[j][2 * m + 1]);
            hi[m] = h0 | (h1 << 16);
            lo[m] = pack_bf16x2(gr[j][2 * m] - bf16_to_f32(h0), gr[j][2 * m + 1] - bf16_to_f32(h1));
          }
          *(u32x2*)&gtl[buf][0][row * GPI + 4 * c4] = u32x2{hi[0], hi[1]};
          *(u32x2*)&gtl[buf][1][row * GPI + 4 * c4] = u32x2{lo[0], lo[1]};
        }
      } else if (q < R * k) {
        const int row = q / k, col = q - row * k;
        const uint32_t h0 = f32_to_bf16(gr[j][0]);
        gtl[buf][0][row * GPI + col] = (uint16_t)h0;
        gtl[buf][1][row * GPI + col] = (uint16_t)f32_to_bf16(gr[j][0] - bf16_to_f32(h0));
      }
    }
  };

  f32x4 acc[CT][KT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int i = 0; i < KT; ++i) acc[ct][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) __attribute__((always_inline)) {
    const uint16_t* hb = (const uint16_t*)ht[buf];
#pragma unroll
    for (int ks = 0; ks < R / 32; ++ks) {
      const int r = 32 * ks + 8 * g + (L >> 2);
      u32x4 bhi[KT], blo[KT];
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        const uint16_t* ph = &gtl[buf][0][r * GPI + 16 * i + 4 * (L & 3)];
        const uint16_t* pl = &gtl[buf][1][r * GPI + 16 * i + 4 * (L & 3)];
        const u32x2 a = lds_read_tr16(ph), b = lds_read_tr16(ph + 4 * GPI);
        const u32x2 x = lds_read_tr16(pl), y = lds_read_tr16(pl + 4 * GPI);
        bhi[i] = u32x4{a[0], a[1], b[0], b[1]};
        blo[i] = u32x4{x[0], x[1], y[0], y[1]};
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const int jl = wave + NW * ct;
        if (jl < tcount) {
          const uint16_t* p = hb + r * (8 * WP) + 16 * jl + 4 * (L & 3);
          const u32x2 a = lds_read_tr16(p), b = lds_read_tr16(p + 4 * 8 * WP);
          const u32x4 af = u32x4{a[0], a[1], b[0], b[1]};
#pragma unroll
          for (int i = 0; i < KT; ++i) {
            acc[ct][i] = mfma16x16x32(af, bhi[i], acc[ct][i]);
            acc[ct][i] = mfma16x16x32(af, blo[i], acc[ct][i]);
          }
        }
      }
    }
  };

  __syncthreads();   // padding zeroed before the first park
  // chunk 0 parked, chunks 1 .. D in flight
  if (nch > 0) {
    load(0, hv[0], gv[0]);
    park(0, hv[0], gv[0]);
#pragma unroll
    for (int j = 1; j <= D; ++j)
      if (nch > j) load(j, hv[j % D], gv[j % D]);
  }
  __syncthreads();
  auto step = [&](int c, auto S) __attribute__((always_inline)) {
    constexpr int sl = decltype(S)::value;      // register set of chunk c + 1
    compute(c & 1);
    if (c + 1 < nch) park((c + 1) & 1, hv[sl], gv[sl]);
    if constexpr (FULL) load(c + 1 + D < nch ? c + 1 + D : nch - 1, hv[sl], gv[sl]);
    else if (c + 1 + D < nch) load(c + 1 + D, hv[sl], gv[sl]);
    __syncthreads();
  };
  for (int c = 0; c < nch; c += D) {
    step(c, std::integral_constant<int, 1 % D>{});
    if (c + 1 < nch) step(c + 1, std::integral_constant<int, 2 % D>{});
    if constexpr (D == 3)
      if (c + 2 < nch) step(c + 2, std::integral_constant<int, 0>{});
  }

  // lane (L, g) of tile (jl, i) holds dZp[col0 + 16 jl + 4g + e][16 i + L]
  float* dst = out + (int64_t)blockIdx.y * din * k;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    const int jl = wave + NW * ct;
    if (jl < tcount) {
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        const int c = 16 * i + L;
        if (c < k) {
#pragma unroll
          for (int e = 0; e < 4; ++e) dst[(int64_t)(col0 + 16 * jl + 4 * g + e) * k + c] = acc[ct][i][e];
        }
      }
    }
  }
}

// ===========================================================================
// Fused backward pass over [N x din], whole tiles and chunks, k = 32 KS2
// (k = 32, 64, 128).  Both gradients of the layer that touch [N x din] come
// from one read of H per chunk of 32 tokens:
//   dZp[cols, :] += H[chunk, cols]^T GT[chunk, :]   (factor gradient: the
//                   MFMA sequence of factor_grad_bf16, from the same LDS tiles)
//   GH[chunk, cols] = GT[chunk, :] Zp[cols, :]^T    (input gradient: the
//                   expansion's sequence, Yt = Zp rows . GT^T with Zp rows
//                   as A fragments held in registers and the GT rows' bf16
//                   hi + lo parts as B fragments read from the LDS tiles)
// so the launch reads H once and writes GH once, side by side, instead of
// one launch writing GH and another reading H.  Per chunk: MFMAs, barrier,
// park the next chunk and write the chunk's GH tile into the LDS tile that
// held its H, barrier, store the tile as whole row pieces (16 bytes per
// thread, 2 TILES pieces per row, non-temporal).  Both results are the same
// bits as the two separate kernels'.
// ===========================================================================
template <int KT, bool NTH, int TILES>
__global__ __launch_bounds__(kFgThreads) void reparam_backward_fused_bf16(
    const uint16_t* __restrict__ H, const float* __restrict__ GT, const uint16_t* __restrict__ Zp,
    uint16_t* __restrict__ GH, float* __restrict__ out, int64_t N, int din, int k, int64_t tps) {
  constexpr int R = kFgRows, NT = kFgThreads, NW = NT / kWave;
  static_assert(TILES % NW == 0 && TILES <= fg_tiles(KT), "whole tiles per wave");
  constexpr int CT = TILES / NW;                       // tiles per wave
  constexpr int HP = 2 * TILES, WP = HP + 1;           // H pieces per row, pitch in pieces
  constexpr int RP = NT / HP;                          // rows per pass
  constexpr int KS2 = (KT + 1) / 2, KW = 32 * KS2;   // k
  constexpr int GPI = KW + 8;                          // GT tile pitch (bf16)
  constexpr int NHP = R / RP;                          // H pieces per thread per chunk
  constexpr int NGQ = (R * KW / 4 + NT - 1) / NT;     // GT pieces per thread per chunk
  static_assert(NT % HP == 0 && R % RP == 0 && R == 32, "piece mapping");
  static_assert(KW == 16 * KT, "k fills its 16-column tiles");
  constexpr int D = KT > 4 ? 2 : kFgDepth;
  __shared__ u32x4 ht[2][R * WP];                      // H chunk, then its GH tile
  __shared__ __align__(16) uint16_t gtl[2][2][R * GPI];   // [buffer][hi / lo][row * GPI + col]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = lane & 15, g = lane >> 4;
  const int col0 = (int)blockIdx.x * 16 * TILES;
  const int64_t t_begin = (int64_t)blockIdx.y * tps;
  const int64_t t_end = min(N, t_begin + tps);
  const int nch = (int)((t_end - t_begin + R - 1) / R);

  const int h = tid % HP, row0 = tid / HP;
  const int64_t rbase = (t_begin + row0) * din + col0 + 8 * h;

  // Zp rows of this wave's tiles: A fragments of the input gradient
  u32x4 za[CT][KS2];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int s = 0; s < KS2; ++s)
      za[ct][s] = *(const u32x4*)(Zp + (int64_t)(col0 + 16 * (wave + NW * ct) + L) * k + 32 * s + 8 * g);

  u32x4 hv[D][NHP];
  f32x4 gv[D][NGQ];
  auto load = [&](int c, u32x4 (&hr)[NHP], f32x4 (&gr)[NGQ]) __attribute__((always_inline)) {
    const int64_t r0 = (int64_t)c * R;
#pragma unroll
    for (int i = 0; i < NHP; ++i) hr[i] = ldg<NTH>(H + rbase + (r0 + RP * i) * din);
#pragma unroll
    for (int j = 0; j < NGQ; ++j) {
      const int q0 = tid + NT * j;
      const int q = q0 < R * (KW / 4) ? q0 : R * (KW / 4) - 1;
      const int row = q / (KW / 4), c4 = q - row * (KW / 4);
      gr[j] = *(const f32x4*)(GT + (t_begin + r0 + row) * KW + 4 * c4);
    }
  };
  auto park = [&](int buf, const u32x4 (&hr)[NHP], const f32x4 (&gr)[NGQ]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NHP; ++i) ht[buf][(row0 + RP * i) * WP + h] = hr[i];
#pragma unroll
    for (int j = 0; j < NGQ; ++j) {
      const int q = tid + NT * j;
      if (q < R * (KW / 4)) {
        const int row = q / (KW / 4), c4 = q - row * (KW / 4);
        uint32_t hi[2], lo[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const uint32_t h0 = f32_to_bf16(gr[j][2 * m]), h1 = f32_to_bf16(gr[j][2 * m + 1]);
          hi[m] = h0 | (h1 << 16);
          lo[m] = pack_bf16x2(gr[j][2 * m] - bf16_to_f32(h0), gr[j][2 * m + 1] - bf16_to_f32(h1));
        }
        *(u32x2*)&gtl[buf][0][row * GPI + 4 * c4] = u32x2{hi[0], hi[1]};
        *(u32x2*)&gtl[buf][1][row * GPI + 4 * c4] = u32x2{lo[0], lo[1]};
      }
    }
  };

  f32x4 acc[CT][KT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int i = 0; i < KT; ++i) acc[ct][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x2 ypk[2][CT];

  auto compute = [&](int buf) __attribute__((always_inline)) {
    const uint16_t* hb = (const uint16_t*)ht[buf];
    // factor gradient: A = H^T (16 din x 32 tokens), B = GT (32 tokens x 16 of k)
    {
      const int r = 8 * g + (L >> 2);
      u32x4 bhi[KT], blo[KT];
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        const uint16_t* ph = &gtl[buf][0][r * GPI + 16 * i + 4 * (L & 3)];
        const uint16_t* pl = &gtl[buf][1][r * GPI + 16 * i + 4 * (L & 3)];
        const u32x2 a = lds_read_tr16(ph), b = lds_read_tr16(ph + 4 * GPI);
        const u32x2 x = lds_read_tr16(pl), y = lds_read_tr16(pl + 4 * GPI);
        bhi[i] = u32x4{a[0], a[1], b[0], b[1]};
        blo[i] = u32x4{x[0], x[1], y[0], y[1]};
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const int jl = wave + NW * ct;
        const uint16_t* p = hb + r * (8 * WP) + 16 * jl + 4 * (L & 3);
        const u32x2 a = lds_read_tr16(p), b = lds_read_tr16(p + 4 * 8 * WP);
        const u32x4 af = u32x4{a[0], a[1], b[0], b[1]};
#pragma unroll
        for (int i = 0; i < KT; ++i) {
          acc[ct][i] = mfma16x16x32(af, bhi[i], acc[ct][i]);
          acc[ct][i] = mfma16x16x32(af, blo[i], acc[ct][i]);
        }
      }
    }
    // input gradient: Yt (16 din x 16 tokens) = Zp rows . GT^T, tokens 16 tt + L
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      u32x4 bh[KS2], bl[KS2];
#pragma unroll
      for (int s = 0; s < KS2; ++s) {
        bh[s] = *(const u32x4*)&gtl[buf][0][(16 * tt + L) * GPI + 32 * s + 8 * g];
        bl[s] = *(const u32x4*)&gtl[buf][1][(16 * tt + L) * GPI + 32 * s + 8 * g];
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS2; ++s) {
          o = mfma16x16x32(za[ct][s], bh[s], o);
          o = mfma16x16x32(za[ct][s], bl[s], o);
        }
        // lane (L, g): GH[token 16 tt + L][din column 16 jl + 4 g + 0 .. 3]
        ypk[tt][ct] = u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
      }
    }
  };

  // chunk 0 parked, chunks 1 .. D in flight (a split without tokens skips all)
  if (nch > 0) {
    load(0, hv[0], gv[0]);
    park(0, hv[0], gv[0]);
#pragma unroll
    for (int j = 1; j <= D; ++j) load(j < nch ? j : nch - 1, hv[j % D], gv[j % D]);
  }
  __syncthreads();
  auto step = [&](int c, auto S) __attribute__((always_inline)) {
    constexpr int sl = decltype(S)::value;      // register set of chunk c + 1
    const int b = c & 1;
    compute(b);
    __syncthreads();   // every wave is done with the chunk's H and GT tiles
    if (c + 1 < nch) park(b ^ 1, hv[sl], gv[sl]);
    load(c + 1 + D < nch ? c + 1 + D : nch - 1, hv[sl], gv[sl]);
    uint16_t* ob = (uint16_t*)ht[b];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
        *(u32x2*)(ob + (16 * tt + L) * (8 * WP) + 16 * (wave + NW * ct) + 4 * g) = ypk[tt][ct];
    __syncthreads();   // the GH tile is complete, the next chunk parked
#pragma unroll
    for (int i = 0; i < NHP; ++i)
      stg<true>(GH + rbase + ((int64_t)c * R + RP * i) * din, ht[b][(row0 + RP * i) * WP + h]);
  };
  for (int c = 0; c < nch; c += D) {
    step(c, std::integral_constant<int, 1 % D>{});
    if (c + 1 < nch) step(c + 1, std::integral_constant<int, 2 % D>{});
    if constexpr (D == 3)
      if (c + 2 < nch) step(c + 2, std::integral_constant<int, 0>{});
  }

  // lane (L, g) of tile (jl, i) holds dZp[col0 + 16 jl + 4g + e][16 i + L]
  float* dst = out + (int64_t)blockIdx.y * din * k;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    const int jl = wave + NW * ct;
#pragma unroll
    for (int i = 0; i < KT; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[(int64_t)(col0 + 16 * jl + 4 * g + e) * k + 16 * i + L] = acc[ct][i][e];
  }
}

// Sum of the S partial results, in split order.
__global__ __launch_bounds__(256) void factor_grad_reduce(const float* __restrict__ ws,
                                                          float* __restrict__ out, int64_t n, int S) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    float s = ws[i];
    for (int j = 1; j < S; ++j) s += ws[(int64_t)j * n + i];
    out[i] = s;
  }
}

// Generic kernel (shapes neither matrix-core kernel takes): one thread per
// output element, fp32 FMA over the tokens in order.
template <typename T>
__global__ __launch_bounds__(256) void factor_grad_generic(const T* __restrict__ H,
                                                           const float* __restrict__ GT,
                                                           float* __restrict__ out, int64_t N,
                                                           int64_t din, int64_t k) {
  for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < din * k;
       o += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = o / k, c = o % k;
    float s = 0.f;
    for (int64_t t = 0; t < N; ++t) s = fmaf(load_as_f32(H + t * din + i), GT[t * k + c], s);
    out[o] = s;
  }
}

static bool factor_grad_uses_mfma(int dtype, int64_t din, int64_t k) {
  return dtype == kBF16 && din % 16 == 0 && din <= INT32_MAX / 2 && k >= 1 && k <= 128;
}

static int fg_tiles_for_k(int64_t k) { return fg_tiles((int)((k + 15) / 16)); }

// Token splits: as many as keep the grid within one round of one block per
// compute unit of an MI355X (256), at least one chunk of tokens per split.
// Depends on (N, din, k) only, so results are the same on every device.
static int64_t factor_grad_splits(int64_t N, int64_t din, int64_t k) {
  const int tiles = fg_tiles_for_k(k);
  const int64_t cb = (din / 16 + tiles - 1) / tiles;
  int64_t S = kFgTargetBlocks / cb;
  const int64_t chunks = (N + kFgRows - 1) / kFgRows;
  S = S > chunks ? chunks : S;
  return S < 1 ? 1 : S;
}

size_t factor_grad_workspace_bytes(int dtype, int64_t N, int64_t din, int64_t k) {
  if (!factor_grad_uses_mfma(dtype, din, k)) return 0;
  const int64_t S = factor_grad_splits(N, din, k);
  return S > 1 ? (size_t)S * (size_t)din * (size_t)k * sizeof(float) : 0;
}

template <int KT>
static hipError_t launch_factor_grad_kt(int64_t N, int din, int k, const void* H, const float* GT,
                                        float* dst, int64_t S, int64_t tps, hipStream_t st) {
  constexpr int TILES = fg_tiles(KT);
  const dim3 grid((unsigned)((din / 16 + TILES - 1) / TILES), (unsigned)S);
  const bool k4 = k % 4 == 0 && ((uintptr_t)GT & 15u) == 0;
  // whole tiles, whole chunks in every split (tps is a multiple of the
  // chunk), and k filling the K slots of its tile bucket
  const bool full = k4 && din % (16 * TILES) == 0 && N % kFgRows == 0 && k == 32 * ((KT + 1) / 2);
  if (full)
    hipLaunchKernelGGL((factor_grad_bf16<KT, true, true, true>), grid, dim3(kFgThreads), 0, st,
                       (const uint16_t*)H, GT, dst, N, din, k, tps);
  else if (k4)
    hipLaunchKernelGGL((factor_grad_bf16<KT, true, false, true>), grid, dim3(kFgThreads), 0, st,
                       (const uint16_t*)H, GT, dst, N, din, k, tps);
  else
    hipLaunchKernelGGL((factor_grad_bf16<KT, false, false, true>), grid, dim3(kFgThreads), 0, st,
                       (const uint16_t*)H, GT, dst, N, din, k, tps);
  return hipGetLastError();
}

// 16-column tiles per block of the fused pass
constexpr int fused_tiles(int kt) { return kt > 4 ? 16 : kFusedTiles; }

bool reparam_backward_fuses(int dtype, int64_t N, int64_t din, int64_t k, const void* H,
                            const float* GT, const void* Zp, const void* GH) {
  const bool wide = k == 32 || k == 64 || k == 128;
  const int64_t cols = 16 * fused_tiles((int)((k + 15) / 16));
  const bool al = (((uintptr_t)H | (uintptr_t)GT | (uintptr_t)Zp | (uintptr_t)GH) & 15u) == 0;
  return dtype == kBF16 && wide && al && N > 0 && N % kFgRows == 0 && din % cols == 0 &&
         din <= INT32_MAX / 2;
}

template <int KT>
static hipError_t launch_fused_kt(int64_t N, int din, int k, const void* H, const float* GT,
                                  const void* Zp, void* GH, float* dst, int64_t S, int64_t tps,
                                  hipStream_t st) {
  constexpr int TILES = fused_tiles(KT);
  const dim3 grid((unsigned)(din / (16 * TILES)), (unsigned)S);
  hipLaunchKernelGGL((reparam_backward_fused_bf16<KT, true, TILES>), grid, dim3(kFgThreads), 0, st,
                     (const uint16_t*)H, GT, (const uint16_t*)Zp, (uint16_t*)GH, dst, N, din, k, tps);
  return hipGetLastError();
}

// Token splits of the fused pass: as factor_grad_splits for its column
// blocks (never more splits than the factor kernel, whose workspace the
// caller sized).
static int64_t fused_splits(int64_t N, int64_t din, int64_t k) {
  const int64_t cb = din / (16 * fused_tiles((int)((k + 15) / 16)));
  int64_t S = kFgTargetBlocks / cb;
  const int64_t chunks = (N + kFgRows - 1) / kFgRows;
  S = S > chunks ? chunks : S;
  S = S < 1 ? 1 : S;
  const int64_t Sf = factor_grad_splits(N, din, k);
  return S < Sf ? S : Sf;
}

hipError_t launch_reparam_backward_fused(int64_t N, int64_t din, int64_t k, const void* H,
                                         const float* GT, const void* Zp, void* GH, float* dZp,
                                         float* ws, hipStream_t st) {
  const int64_t S = fused_splits(N, din, k);
  const int64_t chunks = (N + kFgRows - 1) / kFgRows;
  const int64_t tps = ((chunks + S - 1) / S) * kFgRows;
  float* dst = S > 1 ? ws : dZp;
  hipError_t e;
  if (k == 32) e = launch_fused_kt<2>(N, (int)din, (int)k, H, GT, Zp, GH, dst, S, tps, st);
  else if (k == 64) e = launch_fused_kt<4>(N, (int)din, (int)k, H, GT, Zp, GH, dst, S, tps, st);
  else e = launch_fused_kt<8>(N, (int)din, (int)k, H, GT, Zp, GH, dst, S, tps, st);
  if (e != hipSuccess || S == 1) return e;
  const int64_t n = din * k;
  const unsigned blocks = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(factor_grad_reduce, dim3(blocks), dim3(256), 0, st, ws, dZp, n, (int)S);
  return hipGetLastError();
}

hipError_t launch_factor_grad(int dtype, int64_t N, int64_t din, int64_t k, const void* H,
                              const float* GT, float* dZp, float* ws, hipStream_t st) {
  if (dtype == kF32 && factor_grad_f32_uses_mfma(N, din, k) && ((uintptr_t)H & 15u) == 0 &&
      ((uintptr_t)GT & 15u) == 0)
    return launch_factor_grad_f32(N, din, k, (const float*)H, GT, dZp, st);
  if (factor_grad_uses_mfma(dtype, din, k) && ((uintptr_t)H & 15u) == 0) {
    const int64_t S = factor_grad_splits(N, din, k);
    const int64_t chunks = (N + kFgRows - 1) / kFgRows;
    const int64_t tps = ((chunks + S - 1) / S) * kFgRows;
    float* dst = S > 1 ? ws : dZp;
    hipError_t e;
    const int kt = (int)((k + 15) / 16);
    if (kt <= 2) e = launch_factor_grad_kt<2>(N, (int)din, (int)k, H, GT, dst, S, tps, st);
    else if (kt <= 4) e = launch_factor_grad_kt<4>(N, (int)din, (int)k, H, GT, dst, S, tps, st);
    else e = launch_factor_grad_kt<8>(N, (int)din, (int)k, H, GT, dst, S, tps, st);
    if (e != hipSuccess || S == 1) return e;
    const int64_t n = din * k;
    const unsigned blocks = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
    hipLaunchKernelGGL(factor_grad_reduce, dim3(blocks), dim3(256), 0, st, ws, dZp, n, (int)S);
    return hipGetLastError();
  }
  const int64_t n = din * k;
  const unsigned blocks = (unsigned)((n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536);
  if (dtype == kF32)
    hipLaunchKernelGGL((factor_grad_generic<float>), dim3(blocks), dim3(256), 0, st,
                       (const float*)H, GT, dZp, N, din, k);
  else
    hipLaunchKernelGGL((factor_grad_generic<uint16_t>), dim3(blocks), dim3(256), 0, st,
                       (const uint16_t*)H, GT, dZp, N, din, k);
  return hipGetLastError();
}

}  // namespace ssn

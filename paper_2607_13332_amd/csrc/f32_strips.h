// Column-strip kernel over the columns of float32 matrices (see the comment
// at the kernel): the weight re-projection W <- U (U^T W) and, in its FG
// mode, the reparameterized layer's factor gradient.  Included by the
// translation units that instantiate it (its launcher is explicitly
// instantiated for 1..4 and 5..8 k tiles in two units that compile in
// parallel) and by the one that dispatches.
#pragma once

#include "ssn_device.h"
#include "ssn_launch.h"

#include <type_traits>

namespace ssn {

// ===========================================================================
// Weight re-projection W <- U (U^T W) with float32 storage (the original SSN's
// step after each optimizer update, sections 4.1 and 6.1).  The columns of
// all matrices of a batch form one sequence of 16-column tiles; block b owns
// tpb consecutive tiles (a strip), one block per compute unit.  The 8 waves
// form TW = 8 / RS tile groups of RS waves: wave w = RS tw + rs owns the
// tiles tw, tw + TW, .. of the strip and row share rs (a group's waves are
// consecutive, so they sit on different SIMDs when waves are placed on the
// four SIMDs in turn, and groups with one tile more do not pile onto one
// SIMD).  Few tiles per block (small matrices) thus still keep all four
// SIMDs on the matrix cores.
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
// stored by the block in 16-byte pieces (non-temporal: W is not read
// again).  Columns past a matrix's n (in its last tile) are neither used nor
// stored.
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
  const int tw = wave / RS, rs = wave % RS;
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
          f32x4 s = red[(RS * tw * E + e) * 64 + lane];
#pragma unroll
          for (int r2 = 1; r2 < RS; ++r2) s += red[((RS * tw + r2) * E + e) * 64 + lane];
          tot[i] = s;
        }
      }
      __syncthreads();                          // every partial read
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const int e = rs + RS * i;
        if (e < E && e % CT < NV) red[(RS * tw * E + e) * 64 + lane] = tot[i];
      }
      __syncthreads();
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int v = 0; v < NV; ++v) acc[kt][v] = red[(RS * tw * E + kt * CT + v) * 64 + lane];
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
    // c + 1 is parked orders the stores of chunk c before chunk c + 2 parks.
    // SM >= 0: this thread's pieces 0 .. SM - 1 are stored in every chunk and
    // the others never (so the stores are unconditional and the wait for the
    // next chunk's U operands, issued before them, leaves them in flight;
    // with conditional stores the compiler cannot count them and drains
    // them before the next chunk's MFMAs).  SM < 0: each piece tests itself.
    auto body2 = [&](int c, auto Sc, auto SMc) {
      constexpr int S = decltype(Sc)::value;
      constexpr int SM = decltype(SMc)::value;
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
      if constexpr (SM >= 0) {
#pragma unroll
        for (int i = 0; i < SM; ++i)
          __builtin_nontemporal_store(*(const f32x4*)(ot + op[i].lofs),
                                      (f32x4*)(op[i].ptr + (int64_t)c * R2 * op[i].ld));
      } else {
#pragma unroll
        for (int i = 0; i < NP2; ++i)
          if (op[i].on && c * R2 + op[i].row < d)
            __builtin_nontemporal_store(*(const f32x4*)(ot + op[i].lofs),
                                        (f32x4*)(op[i].ptr + (int64_t)c * R2 * op[i].ld));
      }
    };
    auto pass2 = [&](auto SMc) {
      if constexpr (NV > 0) load_ua(0, ua[0]);
      int c = 0;
      if constexpr (PD == 2) {
        for (; c + 1 < nch2; c += 2) {
          body2(c, std::integral_constant<int, 0>{}, SMc);
          body2(c + 1, std::integral_constant<int, 1>{}, SMc);
        }
      } else if (nch2 > 0) {
        // the first chunk apart: every entry to the loop then has the same
        // stores in flight after the U loads it waits for
        body2(0, std::integral_constant<int, 0>{}, SMc);
        c = 1;
      }
      for (; c < nch2; ++c) body2(c, std::integral_constant<int, 0>{}, SMc);
    };
    // pieces on in every chunk: op[i].on, and the rows of the last chunk
    // inside d (always when d is a multiple of the chunk)
    int ns = 0;
    bool prefix = true;
#pragma unroll
    for (int i = 0; i < NP2; ++i) {
      const bool on = op[i].on && d % R2 == 0;
      prefix = prefix && (on ? ns == i : true);
      ns += on ? 1 : 0;
    }
    if (__all(prefix && ns == NP2)) {
      pass2(std::integral_constant<int, NP2>{});
    } else if (NP2 > 1 && __all(prefix && ns == NP2 - 1)) {
      pass2(std::integral_constant<int, (NP2 > 1 ? NP2 - 1 : 0)>{});
    } else {
      pass2(std::integral_constant<int, -1>{});
    }
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
hipError_t launch_weights_f32_kt(const ColumnBatchF32& cb, const float* U, int d, int k, float* fg_out,
                                 hipStream_t st) {
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

// Explicitly instantiated in f32_strips_a.hip (KT 1..4) and f32_strips_b.hip
// (KT 5..8); the dispatching unit declares them extern.
#define SSN_STRIPS_F32_KT(KT, FG)                                                                 \
  template hipError_t launch_weights_f32_kt<KT, FG>(const ColumnBatchF32&, const float*, int, int, \
                                                    float*, hipStream_t)
#define SSN_STRIPS_F32_KT_EXTERN(KT, FG) extern SSN_STRIPS_F32_KT(KT, FG)

}  // namespace ssn

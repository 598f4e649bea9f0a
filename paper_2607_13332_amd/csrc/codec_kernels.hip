// Stage-boundary codec kernels: compress / gradient projection (contract over
// d) and decompress / gradient expansion (contract over k).
//
// Paper: section 4.1, Eq. (2) -- Z = (X - E[ids]) U, reconstruction with U^T;
// gradients cross the boundary through the same projection (G_Z = G U at the
// receiver, G_Z U^T at the sender).
#include "ssn_device.h"
#include "ssn_launch.h"

#include <type_traits>

namespace ssn {

// ===========================================================================
// compress / project_grad, bf16 storage, MFMA 16x16x32 with fp32 accumulate.
//
// U is [d][k] (k contiguous) and a B fragment needs 8 consecutive d of one
// column, so U is staged per d chunk into LDS already in B-fragment order:
// thread (s, g, n) of the staging pass loads the 8 x KP block
// U[d0+32s+8g .. +7][n*KP .. n*KP+KP-1] and transposes it in registers into
// KP fragments; fragment i carries column n*KP + i.  MFMA N tile i therefore
// produces columns {n*KP + i}, so after the KP tiles each lane holds KP
// consecutive columns of Z per token: contiguous stores.
// ===========================================================================
// Stages one d chunk of U (KS K steps of 32 rows) into LDS in B-fragment
// order for the "contract over d" kernels.  Fragment (K step s, column tile i)
// for lane 16*g + n holds U[32s + 8g .. +7][n*KP + i] (column i of lane
// position n's KP-column block).
//   WIDE (k == 16*KP, KP in {2,4,8}): a task is an 8-row x 8-column block read
//     with 16-byte row loads (one wave instruction covers whole 128-byte rows)
//     that feeds 8/KP lane positions;
//   otherwise a task is the 8-row x KP-column block of one lane position,
//     with per-element bounds predicates when k < 16*KP.
template <int KP, bool KFULL, int KS, int NTHREADS>
struct UStage {
  static constexpr bool WIDE = KFULL && (KP == 2 || KP == 4 || KP == 8);
  static constexpr int NTASK = WIDE ? KS * 8 * KP : KS * kWave;
  static constexpr int TPT = (NTASK + NTHREADS - 1) / NTHREADS;
  static constexpr int UW = WIDE ? 4 : (KP + 1) / 2;
  int srow[TPT], scol[TPT], sidx[TPT];
  bool on[TPT];
  uint32_t w[TPT][8][UW];

  __device__ __forceinline__ void init(int tid) {
#pragma unroll
    for (int q = 0; q < TPT; ++q) {
      const int t = tid + q * NTHREADS;
      on[q] = t < NTASK;
      if constexpr (WIDE) {
        const int sk = t / (8 * KP), rem = t % (8 * KP);
        srow[q] = 32 * sk + 8 * (rem / (2 * KP));
        scol[q] = 8 * (rem % (2 * KP));
        sidx[q] = sk * KP * kWave + 16 * (rem / (2 * KP)) + scol[q] / KP;
      } else {
        srow[q] = 32 * (t >> 6) + 8 * ((t >> 4) & 3);
        scol[q] = (t & 15) * KP;
        sidx[q] = (t >> 6) * KP * kWave + (t & 63);
      }
    }
  }
  __device__ __forceinline__ void load(const uint16_t* __restrict__ U, int64_t row0, int k) {
#pragma unroll
    for (int q = 0; q < TPT; ++q)
      if (on[q]) {
        if constexpr (WIDE) load_block8<8, true>(U, row0 + srow[q], scol[q], k, k, w[q]);
        else load_block8<KP, KFULL>(U, row0 + srow[q], scol[q], k, k, w[q]);
      }
  }
  __device__ __forceinline__ void store(u32x4* lds) const {
#pragma unroll
    for (int q = 0; q < TPT; ++q)
      if (on[q]) {
        if constexpr (WIDE) {
#pragma unroll
          for (int c = 0; c < 8; ++c) lds[sidx[q] + (c % KP) * kWave + c / KP] = block8_column<8>(w[q], c);
        } else {
#pragma unroll
          for (int i = 0; i < KP; ++i) lds[sidx[q] + i * kWave] = block8_column<KP>(w[q], i);
        }
      }
  }
};

constexpr int kCompressKS = 4;                 // K steps (of 32) per d chunk
constexpr int kCompressDC = 32 * kCompressKS;  // d chunk

// ===========================================================================
// compress / project_grad / projected-table compress, many tokens.
//
// Wave w of the block owns 16 consecutive tokens (one MFMA M tile); d is
// walked in chunks of 128 (4 K steps of 32), U staged per chunk by UStage
// (double buffered, one barrier per chunk).  Each wave loads its 16 X rows
// and 16 E[ids] rows for a chunk as 4 instructions of 4 rows x 256 contiguous
// bytes (8 whole 128-byte lines per instruction), parks them in a
// wave-private XOR-swizzled LDS tile, and reads its A fragments from there.
// The embedding subtraction is fused by linearity: X.U and E[ids].U are
// accumulated by identical MFMA sequences into separate fp32 accumulators and
// subtracted once at the end (compress(E[ids]) is exactly zero).
//
// Rows travel DEPTH chunks ahead of the MFMAs in DEPTH register sets.  Within
// a step the next chunk's U is requested before the rows of chunk c + DEPTH:
// loads complete in issue order, so the wait for U at the end of the step
// leaves the younger row loads in flight.  The last DEPTH steps issue no row
// loads (the loop is split so that every load in the main loop is
// unconditional; nch must be a multiple of DEPTH).  ROT: every block starts
// its sweep of d at its own chunk (spreads the concurrent requests of the
// blocks over the columns of the rows).  NTX / NTE: non-temporal loads of the
// activation / embedding rows.
// ===========================================================================
//
// HAS_P (with HAS_E false): Z = X.U - P[ids] with the projected table
// P = E.U (section 4.1: E and U are fixed, so the subtraction commutes with
// the projection); the table rows are subtracted in the epilogue.
template <int KP, bool HAS_E, bool KFULL, int WAVES = 8, int DEPTH = 1, bool NTX = false,
          bool NTE = false, bool ROT = false, int ROTG = 1, bool HAS_P = false>
__global__ __launch_bounds__(64 * WAVES) void compress_rows_bf16(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    float* __restrict__ Z, int64_t N, int d, int k, int64_t V, const float* __restrict__ P,
    uint16_t* __restrict__ Zb, int kz) {
  static_assert(DEPTH >= 1 && DEPTH <= 4, "one to four chunks of rows in flight");
  static_assert(!(HAS_E && HAS_P), "the embedding is subtracted as rows or as projected rows");
  constexpr int KS = 4, DC = 128;
  __shared__ u32x4 lds[2][KS * KP * kWave];      // U B fragments, double buffered
  __shared__ u32x4 tile[WAVES][HAS_E ? 2 : 1][16 * 16];   // [wave][X/E][row * 16 + cell ^ row]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = ((int64_t)blockIdx.x * WAVES + wave) * 16;

  // row-contiguous loads: instruction i covers rows 4i + lane/16, cell lane%16
  const int lc = lane & 15;
  const uint16_t* xr[4];
  const uint16_t* er[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * i + (lane >> 4);
    int64_t t = tok0 + r;
    t = t < N ? t : N - 1;
    xr[i] = X + t * d + 8 * lc;
    er[i] = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * lc : nullptr;
  }
  // HAS_P: the table rows of the epilogue's tokens 4g + j, looked up now so
  // that the end of the kernel waits for one load instead of two
  int64_t prow[HAS_P ? 4 : 1];
  if constexpr (HAS_P) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t tj = tok0 + 4 * g + j;
      prow[j] = tj < N ? clamp_id(ids[tj], V) * kz : 0;
    }
  }
  // blockIdx.y selects one of gridDim.y equal ranges of d (a plain
  // projection with few tokens: the range's partial product goes to rows
  // [blockIdx.y * N, (blockIdx.y + 1) * N) of Z, summed afterwards)
  const int nch = d / DC / (int)gridDim.y;
  const int cbase = (int)blockIdx.y * nch;
  // rotation in units of ROTG chunks (when they divide nch)
  const int rg = (ROTG > 1 && nch % ROTG == 0) ? ROTG : 1;
  const int rot = ROT ? (int)(blockIdx.x % (unsigned)(nch / rg)) * rg : 0;
  auto chunk = [&](int i) { const int x = i + rot; return cbase + (x < nch ? x : x - nch); };

  // DEPTH register sets: step i's rows travel in set i % DEPTH
  u32x4 xv[DEPTH][4], ev[DEPTH][4];
  auto load_rows = [&](int c, u32x4 (&xs)[4], u32x4 (&es)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xs[i] = ldg<NTX>(xr[i] + c * DC);
      if constexpr (HAS_E) es[i] = ldg<NTE>(er[i] + c * DC);
    }
  };
  u32x4* tx = tile[wave][0];
  u32x4* te = tile[wave][HAS_E ? 1 : 0];
  auto park_rows = [&](const u32x4 (&xs)[4], const u32x4 (&es)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + (lane >> 4);
      tx[r * 16 + (lc ^ r)] = xs[i];
      if constexpr (HAS_E) te[r * 16 + (lc ^ r)] = es[i];
    }
  };

  UStage<KP, KFULL, KS, 64 * WAVES> ust;
  ust.init(tid);
  auto load_u = [&](int c) { ust.load(U, (int64_t)c * DC, k); };
  auto store_u = [&](int buf) { ust.store(lds[buf]); };

  f32x4 accX[KP], accE[KP];
#pragma unroll
  for (int i = 0; i < KP; ++i) {
    accX[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    accE[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

#pragma unroll
  for (int j = 0; j < DEPTH; ++j) load_rows(chunk(j), xv[j], ev[j]);
  load_u(chunk(0));
  store_u(0);
  // step i (i % DEPTH == S): park the rows of chunk i, request U of chunk
  // i + 1 and then (LOAD) the rows of chunk i + DEPTH, barrier, MFMAs, stage U.
  auto step = [&](int i, auto Sc, auto Lc) {
    constexpr int S = decltype(Sc)::value;
    constexpr bool LOAD = decltype(Lc)::value;
    park_rows(xv[S], ev[S]);
    load_u(chunk(i + 1 < nch ? i + 1 : i));
    if constexpr (LOAD) load_rows(chunk(i + DEPTH), xv[S], ev[S]);
    __syncthreads();
    const u32x4* fr = lds[i & 1];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int cell = (4 * s + g) ^ n16;
      const u32x4 xa = tx[n16 * 16 + cell];
      u32x4 ea;
      if constexpr (HAS_E) ea = te[n16 * 16 + cell];
      u32x4 bfr[KP];
#pragma unroll
      for (int q = 0; q < KP; ++q) bfr[q] = fr[(s * KP + q) * kWave + lane];
#pragma unroll
      for (int q = 0; q < KP; ++q) {
        accX[q] = mfma16x16x32(xa, bfr[q], accX[q]);
        if constexpr (HAS_E) accE[q] = mfma16x16x32(ea, bfr[q], accE[q]);
      }
    }
    store_u((i + 1) & 1);
  };
  using L1 = std::true_type;
  using L0 = std::false_type;
  for (int i0 = 0; i0 < nch - DEPTH; i0 += DEPTH) {
    step(i0, std::integral_constant<int, 0>{}, L1{});
    if constexpr (DEPTH > 1) step(i0 + 1, std::integral_constant<int, 1 % DEPTH>{}, L1{});
    if constexpr (DEPTH > 2) step(i0 + 2, std::integral_constant<int, 2 % DEPTH>{}, L1{});
    if constexpr (DEPTH > 3) step(i0 + 3, std::integral_constant<int, 3 % DEPTH>{}, L1{});
  }
  {
    const int i0 = nch - DEPTH;
    step(i0, std::integral_constant<int, 0>{}, L0{});
    if constexpr (DEPTH > 1) step(i0 + 1, std::integral_constant<int, 1 % DEPTH>{}, L0{});
    if constexpr (DEPTH > 2) step(i0 + 2, std::integral_constant<int, 2 % DEPTH>{}, L0{});
    if constexpr (DEPTH > 3) step(i0 + 3, std::integral_constant<int, 3 % DEPTH>{}, L0{});
  }

  // lane (n16, g) holds coordinates col0 .. col0 + KP - 1 of tokens
  // tok0 + 4g + j; rows of Z (and P) hold kz of the k columns of U
  const int col0 = n16 * KP;
  bool whole = false;                           // whole 16-byte row pieces
  if constexpr (KFULL && KP % 4 == 0) whole = (kz == k);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t tj = tok0 + 4 * g + j;
    if (tj < N) {
      float v[KP];
#pragma unroll
      for (int i = 0; i < KP; ++i) v[i] = HAS_E ? accX[i][j] - accE[i][j] : accX[i][j];
      if constexpr (HAS_P) {
        const float* pp = P + prow[j] + col0;
        if constexpr (KFULL && KP % 4 == 0) {
          if (whole) {
#pragma unroll
            for (int i = 0; i < KP; i += 4) {
              const f32x4 q = *(const f32x4*)(pp + i);
              v[i] -= q[0]; v[i + 1] -= q[1]; v[i + 2] -= q[2]; v[i + 3] -= q[3];
            }
          }
        }
        if (!whole) {
#pragma unroll
          for (int i = 0; i < KP; ++i)
            if (col0 + i < kz) v[i] -= pp[i];
        }
      }
      if (Zb) {
        // bf16 coordinates: rounded once, to nearest even
        uint16_t* zb = Zb + tj * kz + col0;
        if constexpr (KFULL && KP % 4 == 0) {
          if (whole) {
#pragma unroll
            for (int i = 0; i < KP; i += 4)
              *(u32x2*)(zb + i) = u32x2{pack_bf16x2(v[i], v[i + 1]), pack_bf16x2(v[i + 2], v[i + 3])};
          }
        }
        if (!whole) {
#pragma unroll
          for (int i = 0; i < KP; ++i)
            if (col0 + i < kz) zb[i] = (uint16_t)f32_to_bf16(v[i]);
        }
      } else {
        float* zp = Z + ((int64_t)blockIdx.y * N + tj) * kz + col0;
        if constexpr (KFULL && KP % 4 == 0) {
          if (whole) {
#pragma unroll
            for (int i = 0; i < KP; i += 4) *(f32x4*)(zp + i) = f32x4{v[i], v[i + 1], v[i + 2], v[i + 3]};
          }
        }
        if (!whole) {
#pragma unroll
          for (int i = 0; i < KP; ++i)
            if (col0 + i < kz) zp[i] = v[i];
        }
      }
    }
  }
}

// ===========================================================================
// compress / project_grad / projected-table compress for few tokens.
//
// With N/128 token tiles below the compute-unit count the kernels above leave
// most of the chip idle.  Here a block is 16*TTW tokens x P waves and wave w
// owns the w-th of P equal ranges of d, walked in chunks of 64 (each U
// fragment feeds TTW token tiles).  Everything a wave
// stages is wave-private (no block barrier until the end): its 16 X rows (and
// 16 E[ids] rows) arrive as 8 rows x 128 contiguous bytes per load
// instruction into an XOR-swizzled row tile, and its U rows arrive in a
// padded row-major tile (zero past k).  UM selects how U is staged:
//   0  k % 8 == 0: 16-byte cells of 8 columns;
//   1  any k (rows start only 2-byte aligned): a cell is loaded as the
//      16-byte window at its start rounded down to even; when it is parked
//      the one missing element comes from the next lane's window (a
//      cross-lane shuffle) and a funnel shift realigns it;
//   2  any k: 16-byte pieces of the chunk's contiguous span, scattered
//      element by element.
// Mode 1 moves fewer LDS bytes but issues misaligned loads; which one is
// faster depends on how many token tiles share each U chunk (measured).  A fragments are plain 16-byte LDS reads, U fragments come
// from LDS transpose reads.  Two chunks are in flight in registers.  At the
// end the P partial (X - E[ids]).U results meet in LDS and are summed in wave
// order (deterministic); HAS_P subtracts the projected table rows instead of
// accumulating E[ids].U.
// ===========================================================================
template <int KP, bool HAS_E, bool HAS_P, int UM, int P, int TTW>
__global__ __launch_bounds__(64 * P) __attribute__((amdgpu_waves_per_eu(1, 2))) void compress_split_bf16(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    float* __restrict__ Z, int64_t N, int d, int k, int64_t V, const float* __restrict__ Pt,
    uint16_t* __restrict__ Zb, int kz) {
  static_assert(!(HAS_E && HAS_P), "the embedding is subtracted as rows or as projected rows");
  static_assert(UM >= 0 && UM <= 2, "U staging mode");
  constexpr bool KV = (UM == 0);
  constexpr int DC = 64;                       // d per chunk (two K steps)
  constexpr int KW = 16 * KP;                  // U tile width
  constexpr int UP = KW + 8;                   // U tile pitch (bf16), rows 16-byte aligned
  constexpr int NUL = (DC * KW / 8 + 63) / 64;  // U row cells per lane
  constexpr int NXE = HAS_E ? 2 : 1;
  constexpr int R = 16 * TTW;                  // token rows of a wave
  constexpr int NXL = 2 * TTW;                 // X (and E) pieces per lane
  // per wave: X / E row tiles [R rows x 8 cells] and the U row tile; after
  // the main loop the same memory holds the partial results
  constexpr int XT_BYTES = NXE * R * 8 * 16;
  constexpr int UT_BYTES = DC * UP * 2;
  constexpr int WAVE_BYTES = XT_BYTES + UT_BYTES;
  constexpr int RED_BYTES = TTW * KP * 64 * 16;
  constexpr int SMEM = (P * WAVE_BYTES > P * RED_BYTES) ? P * WAVE_BYTES : P * RED_BYTES;
  __shared__ __align__(16) unsigned char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = (int64_t)blockIdx.x * R;
  // gridDim.y > 1 (plain projections only): block y covers the y-th of
  // gridDim.y equal ranges of d and writes its partial product to
  // Z + y * N * k (summed by a second kernel)
  const int nchp = d / (DC * P * (int)gridDim.y);   // chunks of this wave
  const int c0 = ((int)blockIdx.y * P + wave) * nchp;
  if constexpr (!HAS_E && !HAS_P) Z += (int64_t)blockIdx.y * N * kz;
  // the final sums: thread tid finishes tile-lanes idx = tid + 64 P j; with
  // HAS_P the table values it subtracts there are loaded now, so that their
  // two dependent loads (id, then table row) overlap the main loop
  constexpr int NEP = (TTW * KP * 64 + 64 * P - 1) / (64 * P);
  float pv[HAS_P ? NEP : 1][4];
  if constexpr (HAS_P) {
#pragma unroll
    for (int j = 0; j < NEP; ++j) {
      const int idx = tid + 64 * P * j;
      const int l = idx % 64, ti = idx / 64, i = ti % KP, tt = ti / KP;
      const int col = 16 * i + (l & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t t = tok0 + 16 * tt + 4 * (l >> 4) + e;
        pv[j][e] = (idx < TTW * KP * 64 && col < kz && t < N) ? Pt[clamp_id(ids[t], V) * kz + col] : 0.f;
      }
    }
  }
  u32x4* const xtw = (u32x4*)(smem + wave * WAVE_BYTES);           // [X/E][row * 8 + cell']
  uint16_t* const utw = (uint16_t*)(smem + wave * WAVE_BYTES + XT_BYTES);

  // X / E row pieces: piece q = lane + 64 j is row q/8, 16-byte cell q%8
  const uint16_t* xr[NXL];
  const uint16_t* er[NXL];
#pragma unroll
  for (int j = 0; j < NXL; ++j) {
    const int q = lane + 64 * j;
    int64_t t = tok0 + q / 8;
    t = t < N ? t : N - 1;
    xr[j] = X + t * d + 8 * (q % 8);
    er[j] = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * (q % 8) : nullptr;
  }

  if constexpr (UM == 2) {
    // the span scatter never writes columns k .. KW
    for (int i = lane; i < UT_BYTES / 16; i += 64) ((u32x4*)utw)[i] = u32x4{0u, 0u, 0u, 0u};
  }

  // two register sets: chunk i of this wave travels in set i % 2
  u32x4 xs[2][NXL], es[2][NXL], us[2][NUL];
  auto load = [&](int c, u32x4 (&x)[NXL], u32x4 (&e)[NXL], u32x4 (&u)[NUL]) __attribute__((always_inline)) {
    const int dcol = c * DC;
#pragma unroll
    for (int j = 0; j < NXL; ++j) {
      x[j] = *(const u32x4*)(xr[j] + dcol);
      if constexpr (HAS_E) e[j] = *(const u32x4*)(er[j] + dcol);
    }
#pragma unroll
    for (int i = 0; i < NUL; ++i) {
      const int q = lane + 64 * i;
      if constexpr (UM == 2) {
        // 16-byte piece q of the chunk's contiguous span of DC*k elements
        const bool ok = q < DC * k / 8;
        u[i] = ok ? *(const u32x4*)(U + (int64_t)dcol * k + 8 * q) : u32x4{0u, 0u, 0u, 0u};
      } else {
        const int row = q / (KW / 8), cell = q % (KW / 8);
        const bool ok = q < DC * KW / 8 && 8 * cell < k;
        const int64_t e0 = (int64_t)(dcol + row) * k + 8 * cell;
        if constexpr (KV)
          u[i] = ok ? *(const u32x4*)(U + e0) : u32x4{0u, 0u, 0u, 0u};
        else
          u[i] = ok ? load_bf16x8_even(U, e0, (int64_t)d * k) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto park = [&](const u32x4 (&x)[NXL], const u32x4 (&e)[NXL], const u32x4 (&u)[NUL]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < NXL; ++j) {
      const int q = lane + 64 * j, row = q / 8;
      xtw[row * 8 + ((q % 8) ^ (row & 7))] = x[j];
      if constexpr (HAS_E) xtw[R * 8 + row * 8 + ((q % 8) ^ (row & 7))] = e[j];
    }
#pragma unroll
    for (int i = 0; i < NUL; ++i) {
      const int q = lane + 64 * i;
      if constexpr (UM == 2) {
        // element by element from the span into the padded tile
        if (q < DC * k / 8) {
          const uint32_t w[4] = {u[i][0], u[i][1], u[i][2], u[i][3]};
          int row = (8 * q) / k, col = 8 * q - row * k;
#pragma unroll
          for (int e2 = 0; e2 < 8; ++e2) {
            utw[row * UP + col] = (uint16_t)((e2 & 1) ? (w[e2 >> 1] >> 16) : (w[e2 >> 1] & 0xFFFFu));
            const bool wrap = (col + 1 == k);
            col = wrap ? 0 : col + 1;
            row = wrap ? row + 1 : row;
          }
        }
      } else {
        const int row = q / (KW / 8), cell = q % (KW / 8);
        u32x4 v = u[i];
        if constexpr (UM == 1) {
          // a row's cells sit in consecutive lanes, so the element after this
          // cell's window starts the next lane's window; chunks start at even
          // rows, so row parity and k decide the alignment
          const uint32_t next = __shfl_down(u[i][0], 1);
          v = realign_bf16x8(u[i], next, (row & k & 1) != 0, k - 8 * cell);
        }
        if (q < DC * KW / 8) *(u32x4*)(utw + row * UP + 8 * cell) = v;
      }
    }
  };

  f32x4 accX[TTW][KP], accE[TTW][KP];
#pragma unroll
  for (int tt = 0; tt < TTW; ++tt)
#pragma unroll
    for (int i = 0; i < KP; ++i) {
      accX[tt][i] = f32x4{0.f, 0.f, 0.f, 0.f};
      accE[tt][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  auto compute = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < DC / 32; ++s) {
      const int cell = (4 * s + g) ^ (n16 & 7);
      u32x4 xa[TTW], ea[TTW];
#pragma unroll
      for (int tt = 0; tt < TTW; ++tt) {
        xa[tt] = xtw[(16 * tt + n16) * 8 + cell];
        if constexpr (HAS_E) ea[tt] = xtw[R * 8 + (16 * tt + n16) * 8 + cell];
      }
      const int r = 32 * s + 8 * g + (n16 >> 2);
#pragma unroll
      for (int i = 0; i < KP; ++i) {
        const uint16_t* p = utw + r * UP + 16 * i + 4 * (n16 & 3);
        const u32x2 a = lds_read_tr16(p), b = lds_read_tr16(p + 4 * UP);
        const u32x4 bfr = u32x4{a[0], a[1], b[0], b[1]};
#pragma unroll
        for (int tt = 0; tt < TTW; ++tt) {
          accX[tt][i] = mfma16x16x32(xa[tt], bfr, accX[tt][i]);
          if constexpr (HAS_E) accE[tt][i] = mfma16x16x32(ea[tt], bfr, accE[tt][i]);
        }
      }
    }
  };
  auto step = [&](int i, auto S) __attribute__((always_inline)) {
    constexpr int sl = decltype(S)::value;       // register set of chunk i + 1
    compute();
    if (i + 1 < nchp) park(xs[sl], es[sl], us[sl]);
    if (i + 3 < nchp) load(c0 + i + 3, xs[sl], es[sl], us[sl]);
  };
  load(c0, xs[0], es[0], us[0]);
  park(xs[0], es[0], us[0]);
  if (nchp > 1) load(c0 + 1, xs[1], es[1], us[1]);
  if (nchp > 2) load(c0 + 2, xs[0], es[0], us[0]);
  for (int i = 0; i < nchp; i += 2) {
    step(i, std::integral_constant<int, 1>{});
    if (i + 1 < nchp) step(i + 1, std::integral_constant<int, 0>{});
  }

  // ---- partial results of the P ranges of d, summed in wave order ----
  __syncthreads();                             // the staging tiles become the reduction buffer
  f32x4* const red = (f32x4*)smem;             // [wave][tt][i][lane]
#pragma unroll
  for (int tt = 0; tt < TTW; ++tt)
#pragma unroll
    for (int i = 0; i < KP; ++i)
      red[((wave * TTW + tt) * KP + i) * 64 + lane] = HAS_E ? accX[tt][i] - accE[tt][i] : accX[tt][i];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NEP; ++j) {
    const int idx = tid + 64 * P * j;
    if (idx >= TTW * KP * 64) break;
    const int l = idx % 64, ti = idx / 64, i = ti % KP, tt = ti / KP;
    f32x4 sum = red[ti * 64 + l];
#pragma unroll
    for (int w = 1; w < P; ++w) sum += red[(w * TTW * KP + ti) * 64 + l];
    // lane l of tile (tt, i) holds Z[tok0 + 16 tt + 4 (l/16) + e][16 i + l % 16]
    const int col = 16 * i + (l & 15);
    if (col < kz) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t t = tok0 + 16 * tt + 4 * (l >> 4) + e;
        if (t < N) {
          float v = sum[e];
          if constexpr (HAS_P) v -= pv[j][e];
          if (Zb)
            Zb[t * kz + col] = (uint16_t)f32_to_bf16(v);
          else
            Z[t * kz + col] = v;
        }
      }
    }
  }
}

// ===========================================================================
// decompress / gradient expansion, bf16 storage, MFMA.
//
// Computes Y^T tiles [16 d x 16 tokens] = U_rows [16 d x k] . Z^T [k x 16 tok]
// so that U is used in its natural [d][k] layout (an A fragment is 16
// contiguous bytes of one U row) and Z rows are B fragments.  Z (fp32) is
// split into bf16 hi + lo parts, two MFMAs each, which keeps ~fp32 accuracy.
//
// Block = 4 waves x 16 tokens.  d is walked in 128-wide chunks, every block
// starting at its own rotated offset (spreads concurrent requests over HBM
// channels).  Per chunk the 256 threads stage the chunk's U rows into LDS in
// A-fragment order (double buffered, one barrier per chunk); each wave runs 8
// MFMA tiles for its 16 tokens and parks the fp32 results in a wave-private,
// XOR-swizzled LDS tile [16 tokens x 128 d].  The epilogue then reads that
// tile back row-wise, adds E[ids] (loaded one chunk ahead, 256 contiguous
// bytes of 4 rows per load instruction), rounds once to bf16, and stores 256
// contiguous bytes of 4 rows per instruction.
// ===========================================================================
constexpr int kDecompressDC = 64;

// KM: 0 when k == 32*KS2; 1 when k % 8 == 0 (16-byte rows of U and Z, zero
// groups past k); 2 for any other k: Z is read element by element, and each
// U fragment (8 columns of one row, zero past k) is read as a 4-byte aligned
// window and realigned in registers when it is stored to LDS.
// GZ: the coordinate row of token t is Z[ids[t]] (a gathered table of
// coordinates, e.g. the factored embedding E U^T of section 4.1) instead of
// Z[t]; used without the additive embedding.
template <int KS2, bool HAS_E, int KM, int DC = kDecompressDC, int DSPLIT = 1, int TW = 4,
          bool NTS = false, bool GZ = false, bool NTE = false, int PF = 1, int SG = 1,
          int ROTG = 1>
__global__ __launch_bounds__(64 * TW * DSPLIT) void decompress_mfma_bf16(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    uint16_t* __restrict__ Y, int64_t N, int d, int k, int64_t V,
    const uint16_t* __restrict__ Zb, int kz) {
  static_assert(DC == 64 || DC == 128, "chunk of 64 or 128 d");
  static_assert(KM >= 0 && KM <= 2, "k layout mode");
  static_assert(!(HAS_E && GZ), "gathered coordinates carry no additive embedding");
  constexpr bool KFULL32 = (KM == 0);
  constexpr int NT = DC / 16;                     // MFMA tiles per chunk
  constexpr int FR = NT * KS2 * kWave;            // A fragments per chunk
  constexpr int PT = 64 * TW;                      // stager threads per part
  constexpr int FPT = (FR + PT - 1) / PT;         // staged per thread (last round partial)
  __shared__ u32x4 ufr[2][DSPLIT * FR];           // [buffer][part * FR + fragment]
  __shared__ f32x4 stage[TW * DSPLIT][16 * (DC / 4)];  // [wave][token * DC/4 + cell ^ token]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  // wave = part * TW + token tile: DSPLIT parts of d run side by side
  const int part = DSPLIT == 1 ? 0 : wave / TW;
  const int64_t tok0 = (int64_t)blockIdx.x * (16 * TW) + (wave % TW) * 16;

  // Z^T B fragments of this wave's 16 tokens.  Tokens past N take row N - 1
  // (here and in the epilogue), so their lanes recompute token N - 1 and
  // store the same bytes to the same row: every store is unconditional.
  u32x4 zhi[KS2], zlo[KS2];
  {
    int64_t t = tok0 + n16;
    t = t < N ? t : N - 1;
    // Z rows hold kz coordinates (for the first kz of the k columns of U)
    const int64_t zrow = (GZ ? clamp_id(ids[t], V) : t) * kz;
    // bf16 coordinates when Zb is non-NULL (exact in the hi part; the lo
    // part is zero), else float32 ones from Zc.  Groups of 8 within kz
    // travel as 16-byte loads when the rows are 16-byte aligned, the rest
    // element by element (zero past kz).
    const bool zb16 = Zb != nullptr;
    const bool zvec = KM != 2 && (zb16 ? kz % 8 == 0 : kz % 4 == 0);
    const float* zp = zb16 ? nullptr : Zc + zrow;
    const uint16_t* zq = zb16 ? Zb + zrow : nullptr;
#pragma unroll
    for (int s = 0; s < KS2; ++s) {
      const int c0 = 32 * s + 8 * g;
      float v[8];
      if (zvec && c0 + 8 <= kz) {
        if (zb16) {
          const u32x4 a = *(const u32x4*)(zq + c0);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] = bf16_to_f32(a[e] & 0xFFFFu);
            v[2 * e + 1] = bf16_to_f32(a[e] >> 16);
          }
        } else {
          const f32x4 a = *(const f32x4*)(zp + c0);
          const f32x4 b = *(const f32x4*)(zp + c0 + 4);
          v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
          v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
        }
      } else if (c0 < kz) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[e] = (c0 + e < kz) ? (zb16 ? bf16_to_f32(zq[c0 + e]) : zp[c0 + e]) : 0.f;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;   // the whole group lies past kz
      }
      split_bf16x8(v, zhi[s], zlo[s]);
    }
  }

  // epilogue rows of this lane: LPR lanes per row, each 8 d (16 bytes);
  // RPI = 64 / LPR rows per store instruction, NQ instructions per chunk
  constexpr int LPR = DC / 8, RPI = 64 / LPR, NQ = 16 / RPI;
  const int ec = lane % LPR;
  const uint16_t* erow[NQ];
  uint16_t* yrow[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    int64_t t = tok0 + RPI * q + lane / LPR;
    t = t < N ? t : N - 1;
    yrow[q] = Y + t * d + 8 * ec;
    erow[q] = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * ec : nullptr;
  }

  // U staging: thread tid stages fragments of part tid/PT.  Fragment f ->
  // tile f/(KS2*64), K step (f/64)%KS2, lane position f%64 = 16*g' + m: row
  // 16*tile + m, columns 32*s + 8*g'.
  //  KM == 0 (k == 32*KS2): a chunk's 64 rows are one contiguous span of
  //    64*k elements, so thread piece p = tid%PT + PT*q loads the 16 bytes at
  //    8p of the span (a wave's load covers 1 KB of whole lines) and stores
  //    them to the fragment that holds them (row p/(k/8), 8-column group
  //    p%(k/8)).  Loading each fragment where it sits in U instead (16 rows
  //    x 64 B per wave instruction) measured 6 % slower (8B-stage decompress).
  //  otherwise thread piece p is fragment p itself, loaded from its row.
  // Threads past the last fragment load fragment FR - 1 again and do not
  // store it, and columns past k load column 0 and store zeros, so that the
  // loads, too, are unconditional.
  const int spart = DSPLIT == 1 ? 0 : tid / PT, stid = DSPLIT == 1 ? tid : tid % PT;
  int srow[FPT], scol[FPT], sdst[FPT];
  bool son[FPT];
#pragma unroll
  for (int q = 0; q < FPT; ++q) {
    const int f0 = stid + PT * q;
    son[q] = FR % PT == 0 || f0 < FR;          // compile-time when every thread stores
    const int f = son[q] ? f0 : FR - 1;
    if constexpr (KM == 0) {
      constexpr int GPR = 4 * KS2;                 // 8-column groups per row
      const int r = f / GPR, cg = f % GPR;
      srow[q] = r;
      scol[q] = 8 * cg;
      sdst[q] = ((r >> 4) * KS2 + (cg >> 2)) * kWave + 16 * (cg & 3) + (r & 15);
    } else {
      const int l = f & 63;
      srow[q] = 16 * (f / (KS2 * kWave)) + (l & 15);
      scol[q] = 32 * ((f / kWave) % KS2) + 8 * (l >> 4);
      sdst[q] = f;
    }
  }
  // U fragments travel as 16-byte pieces, or (KM == 2) as unaligned windows
  // that are realigned when they are stored to LDS.  Two register sets:
  // chunk j's fragments travel in set j % 2, loaded two chunks before the
  // chunk that reads them from LDS.
  using UReg = std::conditional_t<KM == 2, Bf16Window, u32x4>;
  UReg ust[2][FPT];
  auto load_u = [&](int c, UReg(&u)[FPT]) {
    if constexpr (KM == 2) {
      // the fragment's 8 columns of one U row
#pragma unroll
      for (int q = 0; q < FPT; ++q)
        u[q] = load_bf16_window(U, (int64_t)(c * DC + srow[q]) * k + (scol[q] < k ? scol[q] : 0),
                                (int64_t)d * k);
    } else {
#pragma unroll
      for (int q = 0; q < FPT; ++q)
        u[q] = *(const u32x4*)(U + (int64_t)(c * DC + srow[q]) * k +
                               (KFULL32 || scol[q] < k ? scol[q] : 0));
    }
  };
  auto store_u = [&](int buf, const UReg(&u)[FPT]) {
#pragma unroll
    for (int q = 0; q < FPT; ++q)
      if (son[q]) {
        u32x4 v;
        if constexpr (KM == 2)
          // chunks start at even rows and fragments at even columns, so row
          // parity and k decide the alignment; zero past k
          v = scol[q] < k ? realign_bf16_window(u[q], (srow[q] & k & 1) != 0, k - scol[q])
                          : u32x4{0u, 0u, 0u, 0u};
        else
          v = (KFULL32 || scol[q] < k) ? u[q] : u32x4{0u, 0u, 0u, 0u};
        ufr[buf][spart * FR + sdst[q]] = v;
      }
  };
  // E rows of chunk j travel in ring slot j % (PF + 1), PF chunks ahead.
  // SG > 1: the packed outputs of SG consecutive chunks are kept in
  // registers and stored together (SG * DC * 2 contiguous bytes per row);
  // then nch must be a multiple of R.
  static_assert(PF == 1 || PF == 3 || PF == 7, "embedding prefetch depth");
  static_assert(SG == 1 || SG == 2 || SG == 4 || SG == 8, "store group");
  constexpr int R = (PF + 1) > SG ? (PF + 1) : SG;   // steps per unrolled group
  u32x4 ering[PF + 1][NQ];
  u32x4 ypk[SG][NQ];
  auto load_e = [&](int c, u32x4(&eo)[NQ]) {
    if constexpr (HAS_E) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) eo[q] = ldg<NTE>(erow[q] + c * DC);
    }
  };

  // blockIdx.y selects one of gridDim.y equal ranges of d (more blocks when
  // there are few tokens); part p of the block walks chunks
  // [(y*DSPLIT + p)*nch, +nch) of that range, rotated per block
  const int nch = d / (DC * DSPLIT * (int)gridDim.y);
  // rotation in units of ROTG chunks (when they divide nch)
  const int rg = (ROTG > 1 && nch % ROTG == 0) ? ROTG : 1;
  const int rot = (int)(blockIdx.x % (unsigned)(nch / rg)) * rg;
  const int pbase = (int)blockIdx.y * DSPLIT;
  auto chunk_of = [&](int p, int i) {
    const int x = i + rot;
    return (pbase + p) * nch + (x < nch ? x : x - nch);
  };
  auto chunk = [&](int i) { return chunk_of(part, i); };
  auto last = [&](int i) { return i < nch ? i : nch - 1; };
  f32x4* st = stage[wave];

  // One chunk, i % R == B.  Order: loads for later chunks (U of chunk i + 2,
  // E of chunk i + PF), barrier, MFMAs, epilogue stores, and only then the
  // LDS store of chunk i + 1's U, whose loads were issued one chunk earlier.
  // Loads and stores share one completion counter, so no wait in a chunk
  // covers the stores that chunk issued.
  auto body = [&](int i, auto Bc) {
    constexpr int B = decltype(Bc)::value;
    constexpr int US = B & 1;
    const int c = chunk(i);
    load_u(chunk_of(spart, last(i + 2)), ust[US]);
    load_e(chunk(last(i + PF)), ering[(B + PF) % (PF + 1)]);
    __syncthreads();
    const u32x4* fr = ufr[US] + part * FR;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS2; ++s) {
        const u32x4 a = fr[(tt * KS2 + s) * kWave + lane];
        acc = mfma16x16x32(a, zhi[s], acc);
        acc = mfma16x16x32(a, zlo[s], acc);
      }
      // lane (token n16, group g) holds d = 16*tt + 4*g + 0..3 of its token
      st[n16 * (DC / 4) + ((4 * tt + g) ^ n16)] = acc;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int tl = RPI * q + lane / LPR;
      const f32x4 a = st[tl * (DC / 4) + ((2 * ec) ^ tl)];
      const f32x4 bb = st[tl * (DC / 4) + ((2 * ec + 1) ^ tl)];
      float v[8] = {a[0], a[1], a[2], a[3], bb[0], bb[1], bb[2], bb[3]};
      if constexpr (HAS_E) {
        const u32x4 e = ering[B % (PF + 1)][q];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          v[2 * m] += lo_bf16(e[m]);
          v[2 * m + 1] += hi_bf16(e[m]);
        }
      }
      const u32x4 y = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                            pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
      if constexpr (SG == 1) stg<NTS>(yrow[q] + c * DC, y);
      else ypk[B % SG][q] = y;
    }
    if constexpr (SG > 1 && B % SG == SG - 1) {
#pragma unroll
      for (int j = 0; j < SG; ++j) {
        const int cj = chunk(i - (SG - 1) + j);
#pragma unroll
        for (int q = 0; q < NQ; ++q) stg<NTS>(yrow[q] + cj * DC, ypk[j][q]);
      }
    }
    store_u(US ^ 1, ust[US ^ 1]);
  };
  auto group = [&](int i0, int n) {   // steps i0 .. i0 + n - 1 (n < R, i0 % R == 0, SG == 1)
    body(i0, std::integral_constant<int, 0>{});
    if (n > 1) body(i0 + 1, std::integral_constant<int, 1>{});
    if constexpr (R > 2) {
      if (n > 2) body(i0 + 2, std::integral_constant<int, 2 % R>{});
      if (n > 3) body(i0 + 3, std::integral_constant<int, 3 % R>{});
    }
    if constexpr (R > 4) {
      if (n > 4) body(i0 + 4, std::integral_constant<int, 4 % R>{});
      if (n > 5) body(i0 + 5, std::integral_constant<int, 5 % R>{});
      if (n > 6) body(i0 + 6, std::integral_constant<int, 6 % R>{});
    }
  };

  load_u(chunk_of(spart, 0), ust[0]);
  load_u(chunk_of(spart, last(1)), ust[1]);
#pragma unroll
  for (int j = 0; j < PF; ++j) load_e(chunk(last(j)), ering[j]);
  store_u(0, ust[0]);
  const int nfull = nch - nch % R;
  for (int i0 = 0; i0 < nfull; i0 += R) {
    body(i0, std::integral_constant<int, 0>{});
    body(i0 + 1, std::integral_constant<int, 1>{});
    if constexpr (R > 2) {
      body(i0 + 2, std::integral_constant<int, 2 % R>{});
      body(i0 + 3, std::integral_constant<int, 3 % R>{});
    }
    if constexpr (R > 4) {
      body(i0 + 4, std::integral_constant<int, 4 % R>{});
      body(i0 + 5, std::integral_constant<int, 5 % R>{});
      body(i0 + 6, std::integral_constant<int, 6 % R>{});
      body(i0 + 7, std::integral_constant<int, 7 % R>{});
    }
  }
  if constexpr (SG == 1) {
    if (nfull < nch) group(nfull, nch - nfull);
  }
}

// ===========================================================================
// Generic kernels: any storage dtype, any d and k.  One wave per token,
// fp32 arithmetic, wavefront reductions.  Used for the shapes the MFMA
// kernels (bf16 here, float32 in f32_kernels.hip) do not tile.
// ===========================================================================
template <typename T, bool HAS_E, bool HAS_P = false>
__global__ __launch_bounds__(256) void compress_generic(
    const T* __restrict__ X, const int32_t* __restrict__ ids, const T* __restrict__ E,
    const T* __restrict__ U, float* __restrict__ Z, int64_t N, int64_t d, int64_t k, int64_t V,
    const float* __restrict__ P, uint16_t* __restrict__ Zb, int64_t kz) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < N; t += nw) {
    const T* xr = X + t * d;
    const T* er = HAS_E ? E + clamp_id(ids[t], V) * d : nullptr;
    // coordinates kc .. kc + 15 of the kz (U rows are k wide)
    for (int64_t kc = 0; kc < kz; kc += 16) {
      float acc[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = 0.f;
      for (int64_t j = lane; j < d; j += 64) {
        const float x = HAS_E ? load_as_f32(xr + j) - load_as_f32(er + j) : load_as_f32(xr + j);
        const T* ur = U + j * k + kc;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (kc + i < kz) acc[i] = fmaf(x, load_as_f32(ur + i), acc[i]);
      }
      float mine = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float s = wave_sum(acc[i]);
        if (lane == i) mine = s;
      }
      if (lane < 16 && kc + lane < kz) {
        if constexpr (HAS_P) mine -= P[clamp_id(ids[t], V) * kz + kc + lane];
        if (Zb)
          Zb[t * kz + kc + lane] = (uint16_t)f32_to_bf16(mine);
        else
          Z[t * kz + kc + lane] = mine;
      }
    }
  }
}

template <typename T, bool HAS_E, bool GZ = false>
__global__ __launch_bounds__(256) void decompress_generic(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids, const T* __restrict__ E,
    const T* __restrict__ U, T* __restrict__ Y, int64_t N, int64_t d, int64_t k, int64_t V,
    const uint16_t* __restrict__ Zb, int64_t kz) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < N; t += nw) {
    const int64_t zrow = (GZ ? clamp_id(ids[t], V) : t) * kz;
    const float* zr = Zb ? nullptr : Zc + zrow;
    const uint16_t* zq = Zb ? Zb + zrow : nullptr;
    const T* er = HAS_E ? E + clamp_id(ids[t], V) * d : nullptr;
    for (int64_t j = lane; j < d; j += 64) {
      float acc = HAS_E ? load_as_f32(er + j) : 0.f;
      const T* ur = U + j * k;
      if (Zb)
        for (int64_t c = 0; c < kz; ++c) acc = fmaf(bf16_to_f32(zq[c]), load_as_f32(ur + c), acc);
      else
        for (int64_t c = 0; c < kz; ++c) acc = fmaf(zr[c], load_as_f32(ur + c), acc);
      store_from_f32(Y + t * d + j, acc);
    }
  }
}

// ===========================================================================
// Launchers.
// ===========================================================================
static inline bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool compress_uses_mfma(int dtype, int64_t d, int64_t k) {
  return dtype == kBF16 && d % kCompressDC == 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

bool decompress_uses_mfma(int dtype, int64_t d, int64_t k) {
  return dtype == kBF16 && d % (2 * kDecompressDC) == 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

// Row-contiguous kernel: 8 waves (128 tokens) per block with a rotated sweep
// of d once N/128 blocks fill the compute units, else 4 waves (64 tokens) in
// the natural order.  The rotation moves in steps of 4 chunks (1 KB of a bf16
// row): on MI355X, start offsets in 256- or 512-byte steps let the blocks'
// concurrent requests collide (measured 1.1-1.8x slower at d = 4096).
// Activation rows are streamed with non-temporal loads; embedding rows keep
// normal caching (repeated ids hit in L2).
// Z = X.U with few tokens: 128-token blocks of the row kernel over S ranges
// of d (grid.y), each writing its partial product to ws [S][N][k].
template <int KP, bool KFULL>
static hipError_t launch_rows_ranges(int64_t N, int d, int k, const void* X, const void* U, float* ws,
                                     int S, hipStream_t st, int kz) {
  const int64_t blocks = (N + 127) / 128;
  hipLaunchKernelGGL((compress_rows_bf16<KP, false, KFULL, 8, 1, true, false, true, 4, false>),
                     dim3((unsigned)blocks, (unsigned)S), dim3(512), 0, st, (const uint16_t*)X,
                     nullptr, nullptr, (const uint16_t*)U, ws, N, d, k, (int64_t)1, nullptr, nullptr, kz);
  return hipGetLastError();
}

template <int KP, bool HAS_E, bool KFULL, bool HAS_P>
static hipError_t launch_compress_rows(int64_t N, int d, int k, int64_t V, const void* X,
                                       const int32_t* ids, const void* E, const void* U, float* Z,
                                       const float* P, hipStream_t st, uint16_t* Zb, int kz) {
  if ((N + 127) / 128 >= device_cu_count()) {
    const int64_t blocks = (N + 127) / 128;
    hipLaunchKernelGGL((compress_rows_bf16<KP, HAS_E, KFULL, 8, 1, true, false, true, 4, HAS_P>),
                       dim3((unsigned)blocks), dim3(512), 0, st, (const uint16_t*)X, ids,
                       (const uint16_t*)E, (const uint16_t*)U, Z, N, d, k, V, P, Zb, kz);
  } else {
    const int64_t blocks = (N + 63) / 64;
    hipLaunchKernelGGL((compress_rows_bf16<KP, HAS_E, KFULL, 4, 1, true, false, false, 1, HAS_P>),
                       dim3((unsigned)blocks), dim3(256), 0, st, (const uint16_t*)X, ids,
                       (const uint16_t*)E, (const uint16_t*)U, Z, N, d, k, V, P, Zb, kz);
  }
  return hipGetLastError();
}

// compress (with the embedding rows), the gradient projection and the
// projected-table compress all use the row-contiguous kernel.
template <int KP, bool HAS_E, bool HAS_P>
static hipError_t launch_compress_kp(int64_t N, int d, int k, int64_t V, const void* X,
                                     const int32_t* ids, const void* E, const void* U, float* Z,
                                     const float* P, hipStream_t st, uint16_t* Zb, int kz) {
  return k == 16 * KP
             ? launch_compress_rows<KP, HAS_E, true, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz)
             : launch_compress_rows<KP, HAS_E, false, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
}

template <bool HAS_E, bool HAS_P>
static hipError_t launch_compress_mfma(int64_t N, int d, int k, int64_t V, const void* X,
                                       const int32_t* ids, const void* E, const void* U, float* Z,
                                       const float* P, hipStream_t st, uint16_t* Zb, int kz) {
  switch ((k + 15) / 16) {
    case 1: return launch_compress_kp<1, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 2: return launch_compress_kp<2, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 3: return launch_compress_kp<3, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 4: return launch_compress_kp<4, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 5: return launch_compress_kp<5, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 6: return launch_compress_kp<6, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    case 7: return launch_compress_kp<7, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
    default: return launch_compress_kp<8, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz);
  }
}

static unsigned generic_blocks(int64_t N) {
  const int64_t want = (N + 3) / 4;
  return (unsigned)(want < 65536 ? want : 65536);
}

// Few tokens: 16-token blocks of P waves that split d (P = 2, 4, 8; P <= 4
// when k > 64, where eight waves' tiles would not fit in LDS).
template <int KP, bool HAS_E, bool HAS_P, int P, int TTW>
static hipError_t launch_split_t(int64_t N, int d, int k, int64_t V, const void* X,
                                 const int32_t* ids, const void* E, const void* U, float* Z,
                                 const float* Pt, hipStream_t st, int S, uint16_t* Zb, int kz) {
  const dim3 grid((unsigned)((N + 16 * TTW - 1) / (16 * TTW)), (unsigned)S);
#define SSN_SPLIT(UM)                                                                           \
  hipLaunchKernelGGL((compress_split_bf16<KP, HAS_E, HAS_P, UM, P, TTW>), grid, dim3(64 * P), 0, \
                     st, (const uint16_t*)X, ids, (const uint16_t*)E, (const uint16_t*)U, Z, N, d, \
                     k, V, Pt, Zb, kz)
  // odd k (measured at d = 5120 and 18432, k = 51): the shuffled windows win
  // when two token tiles share each U chunk, or with eight waves and d up to
  // 8192; otherwise the span scatter, except for compress with eight waves,
  // where the scatter's registers beside the E rows would spill
  if (k % 8 == 0) SSN_SPLIT(0);
  else if constexpr (TTW == 2 || (P == 8 && HAS_E)) SSN_SPLIT(1);
  else if constexpr (P == 8) {
    if (d <= 8192) SSN_SPLIT(1);
    else SSN_SPLIT(2);
  } else SSN_SPLIT(2);
#undef SSN_SPLIT
  return hipGetLastError();
}

template <int KP, bool HAS_E, bool HAS_P>
static hipError_t launch_split_kp(int P, int TTW, int64_t N, int d, int k, int64_t V, const void* X,
                                  const int32_t* ids, const void* E, const void* U, float* Z,
                                  const float* Pt, hipStream_t st, int S, uint16_t* Zb, int kz) {
  if constexpr (KP <= 4) {
    if constexpr (!HAS_E)
      if (P == 8 && TTW == 2)
        return launch_split_t<KP, HAS_E, HAS_P, 8, 2>(N, d, k, V, X, ids, E, U, Z, Pt, st, S, Zb, kz);
    if (P == 8) return launch_split_t<KP, HAS_E, HAS_P, 8, 1>(N, d, k, V, X, ids, E, U, Z, Pt, st, S, Zb, kz);
    if (P == 4 && TTW == 2)
      return launch_split_t<KP, HAS_E, HAS_P, 4, 2>(N, d, k, V, X, ids, E, U, Z, Pt, st, S, Zb, kz);
  }
  if (P >= 4) return launch_split_t<KP, HAS_E, HAS_P, 4, 1>(N, d, k, V, X, ids, E, U, Z, Pt, st, S, Zb, kz);
  return launch_split_t<KP, HAS_E, HAS_P, 2, 1>(N, d, k, V, X, ids, E, U, Z, Pt, st, S, Zb, kz);
}

// When the d-split kernel runs (measured on MI355X at d = 4096 and 5120):
// with k % 8 == 0 the token-parallel kernels win once N/64 (compress) or
// N/128 (projection) blocks fill the chip, above 8192 and 16384 tokens; for
// other k those kernels stage U element by element and the d-split kernel
// wins at every N.
static bool compress_uses_split(int64_t N, int64_t d, int64_t k, bool has_e) {
  if (d % 128 != 0) return false;
  if (k % 8 != 0) return true;
  // The token-parallel kernel stages U in 16-byte row pieces only for k = 32,
  // 64 and 128; for other k it moves a few elements per row and the d-split
  // kernel wins (N = 12288 .. 32768, d = 4096 and 5120: compress 116 -> 61
  // us at k = 40, N = 12288; project_grad 107 -> 57 us at k = 56, N = 32768).
  // For k > 64 it does so only below about 24576 tokens and for an odd
  // number of 16-column tiles (k = 72 and 112: 177 -> 98 us and 217 -> 100
  // us at N = 12288; at k = 96 the token-parallel kernel stays ahead, 67
  // against 99 us, and at 32768 tokens the d-split kernel's four-wave blocks
  // fall behind).
  const int kp = (int)((k + 15) / 16);
  const bool wide = k == 16 * kp && (kp == 2 || kp == 4 || kp == 8);
  if (!wide && (k <= 64 || (kp % 2 == 1 && N <= 24576))) return true;
  return N <= (has_e ? 8192 : 16384);
}

// Shape of a few-token launch: P waves over d, TTW token tiles per wave, S
// ranges of d (grid.y; S > 1 only for plain projections with room for the
// partial products).
struct SplitPlan {
  int P, TTW, S;
};

// compress (E[ids] rows stream beside X): one tile per wave, eight waves
// while that gives about eight waves per compute unit, else four.  k > 64:
// four waves, one tile (LDS).  Projections: two tiles per wave (each U chunk
// staged then feeds 32 tokens, half the U traffic through L2) unless their
// blocks would fill under 60% of the last round on the compute units (a
// unit holds 8/P blocks: two waves per SIMD); for the tile count taken, the
// number of ranges S <= smax whose blocks fill the last round best, fewer
// ranges unless the fill is 5% better; eight waves while the blocks of one
// range fit one round.  P drops where the ranges would not split d into
// whole chunks.  Measured on MI355X (din = 14336 and 18432, k = 51 and 64,
// N = 1000 to 16384), e.g. N = 4096, k = 51: 62 us with one tile, 46 us
// with two tiles in two ranges; N = 3000 without ranges: one tile 58 us,
// two tiles 61 us; N = 6144: two tiles 80 us, 74 us in four ranges.
static SplitPlan split_plan(int64_t N, int d, int k, bool has_e, int smax) {
  if (has_e || k > 64) {
    SplitPlan p{k > 64 ? 4 : (N <= 6144 ? 8 : 4), 1, 1};
    while (p.P > 2 && d % (64 * p.P) != 0) p.P /= 2;
    return p;
  }
  const int64_t cus = device_cu_count();
  auto best_for = [&](int ttw, double& bfill) {
    SplitPlan best{2, 1, 1};
    bfill = 0.0;
    for (int s = 1; s <= smax; ++s) {
      int P = (N + 16 * ttw - 1) / (16 * ttw) <= cus ? 8 : 4;
      while (P > 2 && d % (64 * P * s) != 0) P /= 2;
      if (d % (64 * P * s) != 0) continue;
      const int t = P == 2 ? 1 : ttw;          // two-wave blocks take one tile
      const int64_t blocks = s * ((N + 16 * t - 1) / (16 * t));
      const int64_t slots = cus * (8 / P);
      const int64_t rounds = (blocks + slots - 1) / slots;
      const double fill = (double)blocks / (double)(rounds * slots);
      if (fill > 1.05 * bfill) {
        bfill = fill;
        best = SplitPlan{P, t, s};
      }
    }
    return best;
  };
  double f2, f1;
  const SplitPlan p2 = best_for(2, f2);
  if (f2 >= 0.6) return p2;
  const SplitPlan p1 = best_for(1, f1);
  return f1 > f2 ? p1 : p2;
}

template <bool HAS_E, bool HAS_P>
static hipError_t launch_split(int64_t N, int d, int k, int64_t V, const void* X, const int32_t* ids,
                               const void* E, const void* U, float* Z, const float* Pt,
                               hipStream_t st, const SplitPlan& p, uint16_t* Zb, int kz) {
  if (k <= 32)
    return launch_split_kp<2, HAS_E, HAS_P>(p.P, p.TTW, N, d, k, V, X, ids, E, U, Z, Pt, st, p.S, Zb, kz);
  if (k <= 64)
    return launch_split_kp<4, HAS_E, HAS_P>(p.P, p.TTW, N, d, k, V, X, ids, E, U, Z, Pt, st, p.S, Zb, kz);
  return launch_split_kp<8, HAS_E, HAS_P>(p.P, p.TTW, N, d, k, V, X, ids, E, U, Z, Pt, st, p.S, Zb, kz);
}

// Sum of S partial results [S][n], in range order (deterministic), into out
// (float32) or outb (bf16, rounded once to nearest even).  VEC: n is a
// multiple of 4 and the pointers are aligned for 16-byte partial and output
// pieces (8-byte for bf16), four sums per thread.
template <bool VEC>
__global__ __launch_bounds__(256) void sum_partials(const float* __restrict__ ws,
                                                    float* __restrict__ out,
                                                    uint16_t* __restrict__ outb, int64_t n, int S) {
  constexpr int W = VEC ? 4 : 1;
  for (int64_t i = W * (blockIdx.x * (int64_t)blockDim.x + threadIdx.x); i < n;
       i += (int64_t)W * gridDim.x * blockDim.x) {
    if constexpr (VEC) {
      f32x4 v = *(const f32x4*)(ws + i);
      for (int j = 1; j < S; ++j) v += *(const f32x4*)(ws + (int64_t)j * n + i);
      if (outb)
        *(u32x2*)(outb + i) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      else
        *(f32x4*)(out + i) = v;
    } else {
      float v = ws[i];
      for (int j = 1; j < S; ++j) v += ws[(int64_t)j * n + i];
      if (outb)
        outb[i] = (uint16_t)f32_to_bf16(v);
      else
        out[i] = v;
    }
  }
}

static hipError_t launch_sum_partials(const float* ws, float* out, uint16_t* outb, int64_t n, int S,
                                      hipStream_t st) {
  const bool vec = n % 4 == 0 && al16(ws) && (outb ? ((uintptr_t)outb & 7u) == 0 : al16(out));
  const int64_t per = vec ? 4 * 256 : 256;
  const int64_t blocks = (n + per - 1) / per < 2048 ? (n + per - 1) / per : 2048;
  if (vec)
    hipLaunchKernelGGL(sum_partials<true>, dim3((unsigned)blocks), dim3(256), 0, st, ws, out, outb, n, S);
  else
    hipLaunchKernelGGL(sum_partials<false>, dim3((unsigned)blocks), dim3(256), 0, st, ws, out, outb, n, S);
  return hipGetLastError();
}

// Up[i, c] = U[i, c] for c < k, 0 for k <= c < ldu: the basis with zero
// columns appended, element by element (a once-per-basis copy).
template <typename T>
__global__ __launch_bounds__(256) void pad_basis(const T* __restrict__ U, T* __restrict__ Up,
                                                 int64_t d, int64_t k, int64_t ldu) {
  const int64_t n = d * ldu;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / ldu, c = i - r * ldu;
    Up[i] = c < k ? U[r * k + c] : T(0);
  }
}

hipError_t launch_pad_basis(int dtype, int64_t d, int64_t k, int64_t ldu, const void* U, void* Up,
                            hipStream_t st) {
  const int64_t n = d * ldu;
  const unsigned blocks = (unsigned)((n + 255) / 256 < 16384 ? (n + 255) / 256 : 16384);
  if (dtype == kF32)
    hipLaunchKernelGGL((pad_basis<float>), dim3(blocks), dim3(256), 0, st, (const float*)U,
                       (float*)Up, d, k, ldu);
  else
    hipLaunchKernelGGL((pad_basis<uint16_t>), dim3(blocks), dim3(256), 0, st, (const uint16_t*)U,
                       (uint16_t*)Up, d, k, ldu);
  return hipGetLastError();
}

template <typename T, bool HAS_E, bool HAS_P>
static hipError_t launch_compress_generic(int64_t N, int64_t d, int64_t k, int64_t V, const void* X,
                                          const int32_t* ids, const void* E, const void* U,
                                          float* Z, const float* P, hipStream_t st, uint16_t* Zb,
                                          int64_t kz) {
  hipLaunchKernelGGL((compress_generic<T, HAS_E, HAS_P>), dim3(generic_blocks(N)), dim3(256), 0, st,
                     (const T*)X, ids, (const T*)E, (const T*)U, Z, N, d, k, V, P, Zb, kz);
  return hipGetLastError();
}

// E non-NULL: Z = (X - E[ids]).U; P non-NULL: Z = X.U - P[ids]; neither: Z = X.U.
// Zb non-NULL: the coordinates go to Zb in bf16 (Z unused).
hipError_t launch_compress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const void* X,
                           const int32_t* ids, const void* E, const void* U, float* Z,
                           const float* P, hipStream_t st, uint16_t* Zb, int kzarg) {
  const int64_t kz64 = (kzarg <= 0 || kzarg > k) ? k : kzarg;
  const int kz = (int)(kz64 < 128 ? kz64 : 128);   // the MFMA paths take k <= 128
  const bool has_e = (E != nullptr), has_p = (P != nullptr);
  const void* zout = Zb ? (const void*)Zb : (const void*)Z;
  if (dtype == kF32 && f32_uses_mfma(d, k) && al16(X) && al16(U) && (!has_e || al16(E)))
    return launch_compress_f32(N, d, k, V, (const float*)X, ids, (const float*)E, (const float*)U, Z,
                               P, st, Zb, kz);
  if (compress_uses_mfma(dtype, d, k) && al16(X) && al16(U) && al16(zout) && (!has_e || al16(E)) &&
      (!has_p || al16(P))) {
    if (compress_uses_split(N, d, k, has_e)) {
      const SplitPlan sp = split_plan(N, (int)d, (int)k, has_e, 1);
      if (has_e) return launch_split<true, false>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st, sp, Zb, kz);
      if (has_p) return launch_split<false, true>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st, sp, Zb, kz);
      return launch_split<false, false>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st, sp, Zb, kz);
    }
    if (has_e) return launch_compress_mfma<true, false>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st, Zb, kz);
    if (has_p) return launch_compress_mfma<false, true>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st, Zb, kz);
    return launch_compress_mfma<false, false>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st, Zb, kz);
  }
  if (dtype == kF32) {
    if (has_e) return launch_compress_generic<float, true, false>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz64);
    if (has_p) return launch_compress_generic<float, false, true>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz64);
    return launch_compress_generic<float, false, false>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz64);
  }
  if (has_e) return launch_compress_generic<uint16_t, true, false>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz64);
  if (has_p) return launch_compress_generic<uint16_t, false, true>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz64);
  return launch_compress_generic<uint16_t, false, false>(N, d, k, V, X, ids, E, U, Z, P, st, Zb, kz64);
}

// Z = X.U; with few tokens the few-token kernel may split d into up to
// smax ranges whose partial products go to ws [S][N][k] and are then summed.
// Ranges of d for the row kernel with few tokens: the smallest S <= smax
// dividing the chunk count for which the 128-token blocks of all ranges
// reach one block per compute unit, each range keeping at least 8 chunks
// (0: the token blocks alone fill the chip, or no such S).  Only for the
// widths whose U the row kernel stages as whole 16-byte row pieces (k = 32,
// 64, 128).  Measured on MI355X, N = 4096, k = 64: H Zp over din = 18432 in
// 8 ranges of 18 chunks (forward 60.5 -> 49.4 us with the expansion); G U
// over d = 5120 in 8 ranges of 5 chunks lost to the d-split kernel, and at
// k = 51 the element-wise U staging made the forward 68 -> 94 us.
static int rows_ranges(int64_t N, int64_t d, int64_t k, int smax) {
  const int64_t blocks = (N + 127) / 128, cus = device_cu_count();
  const int nch = (int)(d / kCompressDC);
  const bool wide = k == 32 || k == 64 || k == 128;
  if (!wide || blocks >= cus || d % kCompressDC != 0) return 0;
  for (int S = 2; S <= smax && 8 * S <= nch; ++S)
    if (nch % S == 0 && blocks * S >= cus) return S;
  return 0;
}

hipError_t launch_project_ranges(int dtype, int64_t N, int64_t d, int64_t k, const void* X,
                                 const void* U, float* Z, float* ws, int smax, hipStream_t st,
                                 uint16_t* Zb, int kz) {
  const int kzv = (kz <= 0 || kz > k) ? (int)k : kz;
  const void* zout = Zb ? (const void*)Zb : (const void*)Z;
  auto sum_ranges = [&](int S) { return launch_sum_partials(ws, Z, Zb, N * kzv, S, st); };
  const int rs = (smax > 1 && ws && dtype == kBF16 && k <= 128 && al16(X) && al16(U) && al16(ws) &&
                  d <= INT32_MAX)
                     ? rows_ranges(N, d, k, smax)
                     : 0;
  if (rs > 1) {
    hipError_t e;
    if (k == 32) e = launch_rows_ranges<2, true>(N, (int)d, (int)k, X, U, ws, rs, st, kzv);
    else if (k == 64) e = launch_rows_ranges<4, true>(N, (int)d, (int)k, X, U, ws, rs, st, kzv);
    else e = launch_rows_ranges<8, true>(N, (int)d, (int)k, X, U, ws, rs, st, kzv);
    if (e != hipSuccess) return e;
    return sum_ranges(rs);
  }
  if (smax > 1 && ws && compress_uses_mfma(dtype, d, k) && al16(X) && al16(U) && al16(ws) &&
      al16(zout) && compress_uses_split(N, d, k, false)) {
    const SplitPlan sp = split_plan(N, (int)d, (int)k, false, smax < 4 ? smax : 4);
    if (sp.S > 1) {
      hipError_t e = launch_split<false, false>(N, (int)d, (int)k, 1, X, nullptr, nullptr, U, ws,
                                                nullptr, st, sp, nullptr, kzv);
      if (e != hipSuccess) return e;
      return sum_ranges(sp.S);
    }
  }
  return launch_compress(dtype, N, d, k, 1, X, nullptr, nullptr, U, Z, nullptr, st, Zb, kzv);
}

// 8 token tiles (128 tokens) per block, each of the 8 waves sweeping the
// block's range of d (rotated per block, in steps of one chunk).  When N/128
// blocks fill the compute units the range is all of d; with fewer tokens a
// second grid dimension splits d (a divisor of the chunk count chosen for
// block fill, below; measured at N = 4096 against blocks
// holding two halves of d in 16 waves: expansion 12.0 -> 9.2 us at d = 4096,
// decompress 13.8 -> 13.2 us).  The gradient expansion (no embedding rows to
// gather) stores two chunks at a time (256 contiguous bytes per row) when
// each block's chunk count is even.  The activation rows are written with
// non-temporal stores (streamed out instead of parked dirty in the caches,
// where they slowed the next kernel's reads).
// Ranges of d (grid.y) for `blocks` token blocks over `chunks` chunks of d:
// 1 when the blocks alone reach one per compute unit; else the smallest
// divisor of the chunk count that leaves every block at least two chunks and
// fills at least 90 % of the blocks' last round, else the smallest that
// reaches one block per unit (N = 12288, d = 5120, k = 51: 96 blocks in 5
// ranges 57.9 us, in 4 ranges 64.3 us).
int decompress_grid_split(int64_t blocks, int chunks) {
  const int64_t cus = device_cu_count();
  int gy = 1;
  if (blocks < cus) {
    int first = 0;
    for (int g = 2; g <= chunks; ++g) {
      if (chunks % g != 0 || (blocks * g < cus && g < chunks)) continue;
      if (first == 0) first = g;
      const int64_t b = blocks * g, rounds = (b + cus - 1) / cus;
      if (2 * g <= chunks && 10 * b >= 9 * rounds * cus) {
        gy = g;
        break;
      }
    }
    if (gy == 1) gy = first > 0 ? first : 1;
  }
  return gy;
}

template <int KS2, bool HAS_E, int KM, bool GZ>
static hipError_t launch_decompress_km(int64_t N, int d, int k, int64_t V, const float* Zc,
                                       const int32_t* ids, const void* E, const void* U, void* Y,
                                       hipStream_t st, const uint16_t* Zb, int kz) {
  constexpr int TW = 8;
  const int64_t blocks = (N + 16 * TW - 1) / (16 * TW);
  const int chunks = d / kDecompressDC;
  const int gy = decompress_grid_split(blocks, chunks);
  const dim3 grid((unsigned)blocks, (unsigned)gy);
  if (!HAS_E && (chunks / gy) % 2 == 0)
    hipLaunchKernelGGL((decompress_mfma_bf16<KS2, HAS_E, KM, kDecompressDC, 1, TW, true, GZ, false,
                                             1, 2>),
                       grid, dim3(64 * TW), 0, st, Zc, ids, (const uint16_t*)E, (const uint16_t*)U,
                       (uint16_t*)Y, N, d, k, V, Zb, kz);
  else
    hipLaunchKernelGGL((decompress_mfma_bf16<KS2, HAS_E, KM, kDecompressDC, 1, TW, true, GZ>), grid,
                       dim3(64 * TW), 0, st, Zc, ids, (const uint16_t*)E, (const uint16_t*)U,
                       (uint16_t*)Y, N, d, k, V, Zb, kz);
  return hipGetLastError();
}

template <int KS2, bool HAS_E, bool GZ>
static hipError_t launch_decompress_ks(int64_t N, int d, int k, int64_t V, const float* Zc,
                                       const int32_t* ids, const void* E, const void* U, void* Y,
                                       hipStream_t st, const uint16_t* Zb, int kz) {
  if (k == 32 * KS2) return launch_decompress_km<KS2, HAS_E, 0, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
  if (k % 8 == 0) return launch_decompress_km<KS2, HAS_E, 1, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
  return launch_decompress_km<KS2, HAS_E, 2, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
}

template <bool HAS_E, bool GZ>
static hipError_t launch_decompress_mfma(int64_t N, int d, int k, int64_t V, const float* Zc,
                                         const int32_t* ids, const void* E, const void* U, void* Y,
                                         hipStream_t st, const uint16_t* Zb, int kz) {
  switch ((k + 31) / 32) {
    case 1: return launch_decompress_ks<1, HAS_E, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
    case 2: return launch_decompress_ks<2, HAS_E, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
    case 3: return launch_decompress_ks<3, HAS_E, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
    default: return launch_decompress_ks<4, HAS_E, GZ>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz);
  }
}

template <typename T, bool HAS_E, bool GZ>
static hipError_t launch_decompress_generic(int64_t N, int64_t d, int64_t k, int64_t V,
                                            const float* Zc, const int32_t* ids, const void* E,
                                            const void* U, void* Y, hipStream_t st,
                                            const uint16_t* Zb, int64_t kz) {
  hipLaunchKernelGGL((decompress_generic<T, HAS_E, GZ>), dim3(generic_blocks(N)), dim3(256), 0, st, Zc,
                     ids, (const T*)E, (const T*)U, (T*)Y, N, d, k, V, Zb, kz);
  return hipGetLastError();
}

hipError_t launch_decompress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const float* Zc,
                             const int32_t* ids, const void* E, const void* U, void* Y,
                             bool gather_z, hipStream_t st, const uint16_t* Zb, int kzarg) {
  const int64_t kz64 = (kzarg <= 0 || kzarg > k || gather_z) ? k : kzarg;
  const int kz = (int)(kz64 < 128 ? kz64 : 128);   // the MFMA paths take k <= 128
  const bool has_e = (E != nullptr);
  const void* zin = Zb ? (const void*)Zb : (const void*)Zc;
  if (dtype == kF32 && f32_uses_mfma(d, k) && al16(U) && al16(Y) && (!has_e || al16(E)))
    return launch_decompress_f32(N, d, k, V, Zc, ids, (const float*)E, (const float*)U, (float*)Y,
                                 gather_z, st, Zb, kz);
  if (decompress_uses_mfma(dtype, d, k) && al16(zin) && al16(U) && al16(Y) && (!has_e || al16(E))) {
    if (has_e) return launch_decompress_mfma<true, false>(N, (int)d, (int)k, V, Zc, ids, E, U, Y, st, Zb, kz);
    if (gather_z) return launch_decompress_mfma<false, true>(N, (int)d, (int)k, V, Zc, ids, E, U, Y, st, Zb, kz);
    return launch_decompress_mfma<false, false>(N, (int)d, (int)k, V, Zc, ids, E, U, Y, st, Zb, kz);
  }
  if (dtype == kF32) {
    if (has_e) return launch_decompress_generic<float, true, false>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz64);
    if (gather_z) return launch_decompress_generic<float, false, true>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz64);
    return launch_decompress_generic<float, false, false>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz64);
  }
  if (has_e) return launch_decompress_generic<uint16_t, true, false>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz64);
  if (gather_z) return launch_decompress_generic<uint16_t, false, true>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz64);
  return launch_decompress_generic<uint16_t, false, false>(N, d, k, V, Zc, ids, E, U, Y, st, Zb, kz64);
}

// ===========================================================================
// ids outside [0, V): one block counts them with a grid-free stride loop and
// a fixed-order LDS reduction; thread 0 writes the count (no atomics).
// ===========================================================================
__global__ __launch_bounds__(1024) void check_ids_kernel(const int32_t* __restrict__ ids, int64_t N,
                                                         int64_t V, int64_t* __restrict__ bad) {
  __shared__ int64_t part[1024];
  int64_t cnt = 0;
  for (int64_t i = threadIdx.x; i < N; i += 1024) {
    const int64_t v = ids[i];
    cnt += (v < 0 || v >= V) ? 1 : 0;
  }
  part[threadIdx.x] = cnt;
  __syncthreads();
  for (int h = 512; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) part[threadIdx.x] += part[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) *bad = part[0];
}

hipError_t launch_check_ids(int64_t N, int64_t V, const int32_t* ids, int64_t* bad, hipStream_t st) {
  hipLaunchKernelGGL(check_ids_kernel, dim3(1), dim3(1024), 0, st, ids, N, V, bad);
  return hipGetLastError();
}

}  // namespace ssn

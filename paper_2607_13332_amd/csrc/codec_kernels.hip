// Stage-boundary codec kernels: compress / gradient projection (contract over
// d) and decompress / gradient expansion (contract over k).
//
// Paper: section 4.1, Eq. (2) -- Z = (X - E[ids]) U, reconstruction with U^T,
// and "the backward pass uses the same compression" (G_Z = G U at the
// receiver, G_Z U^T at the sender).
#include "ssn_device.h"
#include "ssn_launch.h"

#include <type_traits>

namespace ssn {

// ===========================================================================
// compress / project_grad, bf16 storage, MFMA 16x16x32 with fp32 accumulate.
//
// Block = 4 waves; wave w owns 16 consecutive tokens (one MFMA M tile).  d is
// walked in chunks of 128 (4 K steps of 32).  For every chunk the 256 threads
// stage that slice of U into LDS already in B-fragment order (double
// buffered, one barrier per chunk), while each wave's X and E[ids] rows go
// from HBM straight into A-fragment registers with 16-byte loads, NBUF-1
// chunks ahead of the MFMAs (a ring of NBUF register buffers).
//
// B-fragment construction (U is [d][k], k contiguous; a fragment needs 8
// consecutive d of one column): thread (s, g, n) of the staging pass loads
// the 8 x KP block U[d0+32s+8g .. +7][n*KP .. n*KP+KP-1] and transposes it in
// registers into KP fragments; fragment i carries column n*KP + i.  MFMA N
// tile i therefore produces columns {n*KP + i}, so after the KP tiles each
// lane holds KP consecutive columns of Z per token: contiguous stores.
//
// The embedding subtraction is fused by linearity: X.U and E[ids].U are
// accumulated by identical MFMA sequences into separate fp32 accumulators
// and subtracted once at the end (compress(E[ids]) is exactly zero).
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

// HAS_P (with HAS_E false): Z = X.U - P[ids], where P = E.U was produced by
// this same kernel with HAS_P false, so that X.U of a row equal to E[id]
// reproduces P[id] bit for bit.
template <int KP, int NBUF, bool HAS_E, bool KFULL, bool ROT = false, bool NT = false,
          int WAVES = 4, int KS = kCompressKS, bool HAS_P = false>
__global__ __launch_bounds__(64 * WAVES) void compress_mfma_bf16(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    float* __restrict__ Z, int64_t N, int d, int k, int64_t V, const float* __restrict__ P) {
  static_assert(!(HAS_E && HAS_P), "the embedding is subtracted as rows or as projected rows");
  constexpr int DC = 32 * KS;
  __shared__ u32x4 lds[2][KS * KP * kWave];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = ((int64_t)blockIdx.x * WAVES + wave) * 16;
  int64_t t = tok0 + n16;
  t = t < N ? t : N - 1;
  const uint16_t* xrow = X + t * d + 8 * g;
  const uint16_t* erow = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * g : nullptr;

  UStage<KP, KFULL, KS, 64 * WAVES> ust;
  ust.init(tid);
  const int nch = d / DC;
  // Each block sweeps the d chunks starting at its own offset: if every wave
  // read the same column range of its rows at the same time, the requests
  // would pile onto a few HBM channels.
  const int rot = ROT ? (int)(blockIdx.x % (unsigned)nch) : 0;
  auto chunk = [&](int c) { const int x = c + rot; return x < nch ? x : x - nch; };

  u32x4 xf[NBUF][KS], ef[NBUF][KS];

  auto load_xe = [&](int c, u32x4(&xo)[KS], u32x4(&eo)[KS]) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      xo[s] = ldg<NT>(xrow + c * DC + 32 * s);
      if constexpr (HAS_E) eo[s] = ldg<NT>(erow + c * DC + 32 * s);
    }
  };
  auto load_u = [&](int c) { ust.load(U, (int64_t)c * DC, k); };
  auto store_u = [&](int buf) { ust.store(lds[buf]); };

  f32x4 accX[KP], accE[KP];
#pragma unroll
  for (int i = 0; i < KP; ++i) {
    accX[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    accE[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

#pragma unroll
  for (int b = 0; b + 1 < NBUF; ++b) load_xe(chunk(b < nch ? b : nch - 1), xf[b], ef[b]);
  load_u(chunk(0));
  store_u(0);

  for (int c0 = 0; c0 < nch; c0 += NBUF) {
#pragma unroll
    for (int b = 0; b < NBUF; ++b) {
      const int c = c0 + b;
      if (c < nch) {
        // U of the next chunk first (it is consumed at the end of this
        // iteration), then X / E of chunk c+NBUF-1 (consumed NBUF-1
        // iterations later): in-order completion lets the staging wait skip
        // the younger X / E loads.
        const int cu = (c + 1 < nch) ? c + 1 : nch - 1;
        load_u(chunk(cu));
        const int pb = (b + NBUF - 1) % NBUF;   // compile-time after unrolling
        const int pf = (c + NBUF - 1 < nch) ? c + NBUF - 1 : nch - 1;
        load_xe(chunk(pf), xf[pb], ef[pb]);
        __syncthreads();
        const u32x4* fr = lds[c & 1];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          u32x4 bfr[KP];
#pragma unroll
          for (int i = 0; i < KP; ++i) bfr[i] = fr[(s * KP + i) * kWave + lane];
#pragma unroll
          for (int i = 0; i < KP; ++i) {
            accX[i] = mfma16x16x32(xf[b][s], bfr[i], accX[i]);
            if constexpr (HAS_E) accE[i] = mfma16x16x32(ef[b][s], bfr[i], accE[i]);
          }
        }
        store_u((c + 1) & 1);
      }
    }
  }

  // ---- epilogue: lane (n16, g) holds Z[tok0+4g+j][n16*KP + i] ----
  const int col0 = n16 * KP;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t tj = tok0 + 4 * g + j;
    if (tj < N) {
      float v[KP];
#pragma unroll
      for (int i = 0; i < KP; ++i) v[i] = HAS_E ? accX[i][j] - accE[i][j] : accX[i][j];
      if constexpr (HAS_P) {
        const float* pp = P + clamp_id(ids[tj], V) * k + col0;
        if constexpr (KFULL && KP % 4 == 0) {
#pragma unroll
          for (int i = 0; i < KP; i += 4) {
            const f32x4 q = *(const f32x4*)(pp + i);
            v[i] -= q[0]; v[i + 1] -= q[1]; v[i + 2] -= q[2]; v[i + 3] -= q[3];
          }
        } else {
#pragma unroll
          for (int i = 0; i < KP; ++i)
            if (col0 + i < k) v[i] -= pp[i];
        }
      }
      float* zp = Z + tj * k + col0;
      if constexpr (KFULL && KP % 4 == 0) {
#pragma unroll
        for (int i = 0; i < KP; i += 4) *(f32x4*)(zp + i) = f32x4{v[i], v[i + 1], v[i + 2], v[i + 3]};
      } else {
#pragma unroll
        for (int i = 0; i < KP; ++i)
          if (col0 + i < k) zp[i] = v[i];
      }
    }
  }
}

// ===========================================================================
// compress / project_grad, variant with row-contiguous activation loads.
//
// Same MFMA scheme as compress_mfma_bf16 (U staged per 128-wide d chunk in
// B-fragment order, X.U and E[ids].U in separate fp32 accumulators), but each
// wave loads its 16 X rows and 16 E[ids] rows for a chunk as 4 instructions
// of 4 rows x 256 contiguous bytes (8 whole 128-byte lines per instruction,
// instead of 16 half lines), parks them in a wave-private XOR-swizzled LDS
// tile, and reads its A fragments from there.  The next chunk's rows are
// loaded into registers while the current chunk computes.
// ===========================================================================
template <int KP, bool HAS_E, bool KFULL, int WAVES = 8, int DEPTH = 1>
__global__ __launch_bounds__(64 * WAVES) void compress_rows_bf16(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    float* __restrict__ Z, int64_t N, int d, int k, int64_t V) {
  static_assert(DEPTH == 1 || DEPTH == 2, "one or two chunks of rows in flight");
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
  // DEPTH register sets: chunk c travels in set c % DEPTH
  u32x4 xv[DEPTH][4], ev[DEPTH][4];
  auto load_rows = [&](int c, u32x4 (&xs)[4], u32x4 (&es)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xs[i] = *(const u32x4*)(xr[i] + c * DC);
      if constexpr (HAS_E) es[i] = *(const u32x4*)(er[i] + c * DC);
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

  const int nch = d / DC;
#pragma unroll
  for (int j = 0; j < DEPTH; ++j)
    if (j < nch) load_rows(j, xv[j], ev[j]);
  load_u(0);
  store_u(0);
  auto step = [&](int c, auto S) {
    constexpr int s0 = decltype(S)::value;       // == c % DEPTH
    park_rows(xv[s0], ev[s0]);
    if (c + DEPTH < nch) load_rows(c + DEPTH, xv[s0], ev[s0]);
    load_u(c + 1 < nch ? c + 1 : c);
    __syncthreads();
    const u32x4* fr = lds[c & 1];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int cell = (4 * s + g) ^ n16;
      const u32x4 xa = tx[n16 * 16 + cell];
      u32x4 ea;
      if constexpr (HAS_E) ea = te[n16 * 16 + cell];
      u32x4 bfr[KP];
#pragma unroll
      for (int i = 0; i < KP; ++i) bfr[i] = fr[(s * KP + i) * kWave + lane];
#pragma unroll
      for (int i = 0; i < KP; ++i) {
        accX[i] = mfma16x16x32(xa, bfr[i], accX[i]);
        if constexpr (HAS_E) accE[i] = mfma16x16x32(ea, bfr[i], accE[i]);
      }
    }
    store_u((c + 1) & 1);
  };
  for (int c = 0; c < nch; c += DEPTH) {
    step(c, std::integral_constant<int, 0>{});
    if constexpr (DEPTH == 2)
      if (c + 1 < nch) step(c + 1, std::integral_constant<int, 1>{});
  }

  const int col0 = n16 * KP;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t tj = tok0 + 4 * g + j;
    if (tj < N) {
      float v[KP];
#pragma unroll
      for (int i = 0; i < KP; ++i) v[i] = HAS_E ? accX[i][j] - accE[i][j] : accX[i][j];
      float* zp = Z + tj * k + col0;
      if constexpr (KFULL && KP % 4 == 0) {
#pragma unroll
        for (int i = 0; i < KP; i += 4) *(f32x4*)(zp + i) = f32x4{v[i], v[i + 1], v[i + 2], v[i + 3]};
      } else {
#pragma unroll
        for (int i = 0; i < KP; ++i)
          if (col0 + i < k) zp[i] = v[i];
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

template <int KS2, bool HAS_E, bool KFULL32, int DC = kDecompressDC, int PF = 1, int DSPLIT = 1,
          int TW = 4, bool NTS = false>
__global__ __launch_bounds__(64 * TW * DSPLIT) void decompress_mfma_bf16(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    uint16_t* __restrict__ Y, int64_t N, int d, int k, int64_t V) {
  static_assert(DC == 64 || DC == 128, "chunk of 64 or 128 d");
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
  const int part = wave / TW;
  const int64_t tok0 = (int64_t)blockIdx.x * (16 * TW) + (wave % TW) * 16;

  // Z^T B fragments of this wave's 16 tokens
  u32x4 zhi[KS2], zlo[KS2];
  {
    int64_t t = tok0 + n16;
    t = t < N ? t : N - 1;
    const float* zp = Zc + t * k;
#pragma unroll
    for (int s = 0; s < KS2; ++s) {
      const int c0 = 32 * s + 8 * g;
      float v[8];
      if (KFULL32 || c0 + 8 <= k) {
        const f32x4 a = *(const f32x4*)(zp + c0);
        const f32x4 b = *(const f32x4*)(zp + c0 + 4);
        v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
        v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;   // k % 8 == 0 on this path
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
  bool ok[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    int64_t t = tok0 + RPI * q + lane / LPR;
    ok[q] = t < N;
    t = t < N ? t : N - 1;
    yrow[q] = Y + t * d + 8 * ec;
    erow[q] = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * ec : nullptr;
  }

  // U staging: thread tid stages fragments of part tid/PT; fragment
  // f = tid%PT + PT*q -> tile f/(KS2*64), K step (f/64)%KS2, lane position
  // f%64 = 16*g' + m: row 16*tile + m, columns 32*s + 8*g'
  const int spart = tid / PT, stid = tid % PT;
  int srow[FPT], scol[FPT];
#pragma unroll
  for (int q = 0; q < FPT; ++q) {
    const int f = stid + PT * q;
    const int l = f & 63;
    srow[q] = 16 * (f / (KS2 * kWave)) + (l & 15);
    scol[q] = 32 * ((f / kWave) % KS2) + 8 * (l >> 4);
  }
  u32x4 ust[FPT];
  auto load_u = [&](int c) {
#pragma unroll
    for (int q = 0; q < FPT; ++q)
      if (stid + PT * q < FR)
        ust[q] = (KFULL32 || scol[q] < k)
                     ? *(const u32x4*)(U + (int64_t)(c * DC + srow[q]) * k + scol[q])
                     : u32x4{0u, 0u, 0u, 0u};
  };
  auto store_u = [&](int buf) {
#pragma unroll
    for (int q = 0; q < FPT; ++q)
      if (stid + PT * q < FR) ufr[buf][spart * FR + stid + PT * q] = ust[q];
  };
  u32x4 ering[PF + 1][NQ];
  auto load_e = [&](int c, u32x4(&eo)[NQ]) {
    if constexpr (HAS_E) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) eo[q] = *(const u32x4*)(erow[q] + c * DC);
    }
  };

  // part p walks chunks [p*nch, (p+1)*nch) of d (nch per part), rotated
  const int nch = d / (DC * DSPLIT);
  const int rot = (int)(blockIdx.x % (unsigned)nch);
  auto chunk_of = [&](int p, int i) { const int x = i + rot; return p * nch + (x < nch ? x : x - nch); };
  auto chunk = [&](int i) { return chunk_of(part, i); };
  f32x4* st = stage[wave];

  // the stager threads of part spart load that part's chunks of U
  auto load_u_part = [&](int i) { load_u(chunk_of(spart, i)); };

  load_u_part(0);
  store_u(0);
#pragma unroll
  for (int b = 0; b < PF; ++b) load_e(chunk(b < nch ? b : nch - 1), ering[b]);
  for (int i0 = 0; i0 < nch; i0 += PF + 1) {
#pragma unroll
    for (int b = 0; b <= PF; ++b) {
      const int i = i0 + b;
      if (i < nch) {
        const int c = chunk(i);
        load_u_part(i + 1 < nch ? i + 1 : i);
        // E of chunk i + PF into the ring slot freed by chunk i - 1
        load_e(chunk(i + PF < nch ? i + PF : nch - 1), ering[(b + PF) % (PF + 1)]);
        __syncthreads();
        const u32x4* fr = ufr[i & 1] + part * FR;
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
            const u32x4 e = ering[b][q];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              v[2 * m] += lo_bf16(e[m]);
              v[2 * m + 1] += hi_bf16(e[m]);
            }
          }
          if (ok[q])
            stg<NTS>(yrow[q] + c * DC, u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                             pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])});
        }
        store_u((i + 1) & 1);
      }
    }
  }
}

// ===========================================================================
// Generic kernels: any storage dtype, any d and k.  One wave per token,
// fp32 arithmetic, wavefront reductions.  Used for fp32 storage and for shapes
// the MFMA kernels do not tile.
// ===========================================================================
template <typename T, bool HAS_E, bool HAS_P = false>
__global__ __launch_bounds__(256) void compress_generic(
    const T* __restrict__ X, const int32_t* __restrict__ ids, const T* __restrict__ E,
    const T* __restrict__ U, float* __restrict__ Z, int64_t N, int64_t d, int64_t k, int64_t V,
    const float* __restrict__ P) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < N; t += nw) {
    const T* xr = X + t * d;
    const T* er = HAS_E ? E + clamp_id(ids[t], V) * d : nullptr;
    for (int64_t kc = 0; kc < k; kc += 16) {
      float acc[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = 0.f;
      for (int64_t j = lane; j < d; j += 64) {
        const float x = HAS_E ? load_as_f32(xr + j) - load_as_f32(er + j) : load_as_f32(xr + j);
        const T* ur = U + j * k + kc;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (kc + i < k) acc[i] = fmaf(x, load_as_f32(ur + i), acc[i]);
      }
      float mine = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float s = wave_sum(acc[i]);
        if (lane == i) mine = s;
      }
      if (lane < 16 && kc + lane < k) {
        if constexpr (HAS_P) mine -= P[clamp_id(ids[t], V) * k + kc + lane];
        Z[t * k + kc + lane] = mine;
      }
    }
  }
}

template <typename T, bool HAS_E>
__global__ __launch_bounds__(256) void decompress_generic(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids, const T* __restrict__ E,
    const T* __restrict__ U, T* __restrict__ Y, int64_t N, int64_t d, int64_t k, int64_t V) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < N; t += nw) {
    const float* zr = Zc + t * k;
    const T* er = HAS_E ? E + clamp_id(ids[t], V) * d : nullptr;
    for (int64_t j = lane; j < d; j += 64) {
      float acc = HAS_E ? load_as_f32(er + j) : 0.f;
      const T* ur = U + j * k;
      for (int64_t c = 0; c < k; ++c) acc = fmaf(zr[c], load_as_f32(ur + c), acc);
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
  return dtype == kBF16 && d % (2 * kDecompressDC) == 0 && d <= INT32_MAX && k % 8 == 0 && k >= 8 && k <= 128;
}

template <int KP, bool HAS_E, bool KFULL, int WAVES, int KS, bool HAS_P>
static hipError_t launch_compress_v(int64_t N, int d, int k, int64_t V, const void* X,
                                    const int32_t* ids, const void* E, const void* U, float* Z,
                                    const float* P, hipStream_t st) {
  const int64_t blocks = (N + 16 * WAVES - 1) / (16 * WAVES);
  hipLaunchKernelGGL((compress_mfma_bf16<KP, 1, HAS_E, KFULL, false, false, WAVES, KS, HAS_P>),
                     dim3((unsigned)blocks), dim3(64 * WAVES), 0, st, (const uint16_t*)X, ids,
                     (const uint16_t*)E, (const uint16_t*)U, Z, N, d, k, V, P);
  return hipGetLastError();
}

template <int KP, bool KFULL>
static hipError_t launch_compress_rows(int64_t N, int d, int k, int64_t V, const void* X,
                                       const int32_t* ids, const void* E, const void* U, float* Z,
                                       hipStream_t st) {
  constexpr int WAVES = 4;
  const int64_t blocks = (N + 16 * WAVES - 1) / (16 * WAVES);
  hipLaunchKernelGGL((compress_rows_bf16<KP, true, KFULL, WAVES>), dim3((unsigned)blocks),
                     dim3(64 * WAVES), 0, st, (const uint16_t*)X, ids, (const uint16_t*)E,
                     (const uint16_t*)U, Z, N, d, k, V);
  return hipGetLastError();
}

// compress (with the embedding rows) uses the row-contiguous variant; the
// gradient projection and the projected-table compress (one activation
// stream) the direct-fragment variant with 8 waves (128 tokens) per block
// sharing each staged slice of U, in 256-d chunks when d allows, else 128.
// The table build (P = E.U) is a gradient-projection launch, so both sides of
// the projected-table compress take the same instantiation.
template <int KP, bool HAS_E, bool HAS_P>
static hipError_t launch_compress_kp(int64_t N, int d, int k, int64_t V, const void* X,
                                     const int32_t* ids, const void* E, const void* U, float* Z,
                                     const float* P, hipStream_t st) {
  const bool kfull = (k == 16 * KP);
  if constexpr (HAS_E)
    return kfull ? launch_compress_rows<KP, true>(N, d, k, V, X, ids, E, U, Z, st)
                 : launch_compress_rows<KP, false>(N, d, k, V, X, ids, E, U, Z, st);
  if (d % 256 == 0)
    return kfull ? launch_compress_v<KP, HAS_E, true, 8, 8, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st)
                 : launch_compress_v<KP, HAS_E, false, 8, 8, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
  return kfull ? launch_compress_v<KP, HAS_E, true, 8, 4, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st)
               : launch_compress_v<KP, HAS_E, false, 8, 4, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
}

template <bool HAS_E, bool HAS_P>
static hipError_t launch_compress_mfma(int64_t N, int d, int k, int64_t V, const void* X,
                                       const int32_t* ids, const void* E, const void* U, float* Z,
                                       const float* P, hipStream_t st) {
  switch ((k + 15) / 16) {
    case 1: return launch_compress_kp<1, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    case 2: return launch_compress_kp<2, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    case 3: return launch_compress_kp<3, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    case 4: return launch_compress_kp<4, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    case 5: return launch_compress_kp<5, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    case 6: return launch_compress_kp<6, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    case 7: return launch_compress_kp<7, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
    default: return launch_compress_kp<8, HAS_E, HAS_P>(N, d, k, V, X, ids, E, U, Z, P, st);
  }
}

static unsigned generic_blocks(int64_t N) {
  const int64_t want = (N + 3) / 4;
  return (unsigned)(want < 65536 ? want : 65536);
}

template <typename T, bool HAS_E, bool HAS_P>
static hipError_t launch_compress_generic(int64_t N, int64_t d, int64_t k, int64_t V, const void* X,
                                          const int32_t* ids, const void* E, const void* U,
                                          float* Z, const float* P, hipStream_t st) {
  hipLaunchKernelGGL((compress_generic<T, HAS_E, HAS_P>), dim3(generic_blocks(N)), dim3(256), 0, st,
                     (const T*)X, ids, (const T*)E, (const T*)U, Z, N, d, k, V, P);
  return hipGetLastError();
}

// E non-NULL: Z = (X - E[ids]).U; P non-NULL: Z = X.U - P[ids]; neither: Z = X.U.
hipError_t launch_compress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const void* X,
                           const int32_t* ids, const void* E, const void* U, float* Z,
                           const float* P, hipStream_t st) {
  const bool has_e = (E != nullptr), has_p = (P != nullptr);
  if (compress_uses_mfma(dtype, d, k) && al16(X) && al16(U) && al16(Z) && (!has_e || al16(E)) &&
      (!has_p || al16(P))) {
    if (has_e) return launch_compress_mfma<true, false>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st);
    if (has_p) return launch_compress_mfma<false, true>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st);
    return launch_compress_mfma<false, false>(N, (int)d, (int)k, V, X, ids, E, U, Z, P, st);
  }
  if (dtype == kF32) {
    if (has_e) return launch_compress_generic<float, true, false>(N, d, k, V, X, ids, E, U, Z, P, st);
    if (has_p) return launch_compress_generic<float, false, true>(N, d, k, V, X, ids, E, U, Z, P, st);
    return launch_compress_generic<float, false, false>(N, d, k, V, X, ids, E, U, Z, P, st);
  }
  if (has_e) return launch_compress_generic<uint16_t, true, false>(N, d, k, V, X, ids, E, U, Z, P, st);
  if (has_p) return launch_compress_generic<uint16_t, false, true>(N, d, k, V, X, ids, E, U, Z, P, st);
  return launch_compress_generic<uint16_t, false, false>(N, d, k, V, X, ids, E, U, Z, P, st);
}

// 8 token tiles (128 tokens) x 2 halves of d per block (16 waves); the
// activation rows are written with non-temporal stores (streamed out instead
// of parked dirty in the caches, where they slowed the next kernel's reads)
template <int KS2, bool HAS_E>
static hipError_t launch_decompress_ks(int64_t N, int d, int k, int64_t V, const float* Zc,
                                       const int32_t* ids, const void* E, const void* U, void* Y,
                                       hipStream_t st) {
  constexpr int TW = 8, DS = 2;
  const int64_t blocks = (N + 16 * TW - 1) / (16 * TW);
  if (k == 32 * KS2)
    hipLaunchKernelGGL((decompress_mfma_bf16<KS2, HAS_E, true, kDecompressDC, 1, DS, TW, true>),
                       dim3((unsigned)blocks), dim3(64 * TW * DS), 0, st, Zc, ids,
                       (const uint16_t*)E, (const uint16_t*)U, (uint16_t*)Y, N, d, k, V);
  else
    hipLaunchKernelGGL((decompress_mfma_bf16<KS2, HAS_E, false, kDecompressDC, 1, DS, TW, true>),
                       dim3((unsigned)blocks), dim3(64 * TW * DS), 0, st, Zc, ids,
                       (const uint16_t*)E, (const uint16_t*)U, (uint16_t*)Y, N, d, k, V);
  return hipGetLastError();
}

template <bool HAS_E>
static hipError_t launch_decompress_mfma(int64_t N, int d, int k, int64_t V, const float* Zc,
                                         const int32_t* ids, const void* E, const void* U, void* Y,
                                         hipStream_t st) {
  switch ((k + 31) / 32) {
    case 1: return launch_decompress_ks<1, HAS_E>(N, d, k, V, Zc, ids, E, U, Y, st);
    case 2: return launch_decompress_ks<2, HAS_E>(N, d, k, V, Zc, ids, E, U, Y, st);
    case 3: return launch_decompress_ks<3, HAS_E>(N, d, k, V, Zc, ids, E, U, Y, st);
    default: return launch_decompress_ks<4, HAS_E>(N, d, k, V, Zc, ids, E, U, Y, st);
  }
}

hipError_t launch_decompress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const float* Zc,
                             const int32_t* ids, const void* E, const void* U, void* Y,
                             hipStream_t st) {
  const bool has_e = (E != nullptr);
  if (decompress_uses_mfma(dtype, d, k) && al16(Zc) && al16(U) && al16(Y) && (!has_e || al16(E))) {
    return has_e ? launch_decompress_mfma<true>(N, (int)d, (int)k, V, Zc, ids, E, U, Y, st)
                 : launch_decompress_mfma<false>(N, (int)d, (int)k, V, Zc, ids, E, U, Y, st);
  }
  const unsigned nb = generic_blocks(N);
  if (dtype == kF32) {
    if (has_e)
      hipLaunchKernelGGL((decompress_generic<float, true>), dim3(nb), dim3(256), 0, st, Zc, ids,
                         (const float*)E, (const float*)U, (float*)Y, N, d, k, V);
    else
      hipLaunchKernelGGL((decompress_generic<float, false>), dim3(nb), dim3(256), 0, st, Zc, ids,
                         (const float*)E, (const float*)U, (float*)Y, N, d, k, V);
  } else {
    if (has_e)
      hipLaunchKernelGGL((decompress_generic<uint16_t, true>), dim3(nb), dim3(256), 0, st, Zc, ids,
                         (const uint16_t*)E, (const uint16_t*)U, (uint16_t*)Y, N, d, k, V);
    else
      hipLaunchKernelGGL((decompress_generic<uint16_t, false>), dim3(nb), dim3(256), 0, st, Zc, ids,
                         (const uint16_t*)E, (const uint16_t*)U, (uint16_t*)Y, N, d, k, V);
  }
  return hipGetLastError();
}

}  // namespace ssn

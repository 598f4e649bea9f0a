// Original-SSN weight re-projection W <- U (U^T W), in place.
//
// Paper: section 4.1 (the original SSN stores each output projection at full
// width and projects it back into the subspace after every optimizer step)
// and section 6.1 (re-projection happens after the optimizer step, outside the
// computational graph).  With PyTorch's [out = d, in = n] layout the rows of
// W are the constrained index, so each column w of W maps to U U^T w.
#include "ssn_device.h"
#include "ssn_launch.h"

#include <atomic>
#include <type_traits>

namespace ssn {

struct PanelBatch {
  uint16_t* W[kMaxBatch];
  int32_t n[kMaxBatch];
  int32_t first_panel[kMaxBatch + 1];
  int32_t count;
};

// ===========================================================================
// Fused single-pass kernel, bf16 storage, MFMA.  One block owns a 64-column
// panel of one matrix over all d rows:
//   pass 1  T = U^T W_panel  (k x 64, fp32): the 4 waves split the d rows,
//           each wave forms U^T and W fragments from 8-row register
//           transposes (no LDS staging), and the 4 partial T are summed in
//           LDS in a fixed order (deterministic);
//   pass 2  W_panel = U T: T^T is split into bf16 hi + lo fragments held in
//           registers, U rows are read in their natural layout, and each lane
//           stores 16 consecutive columns of one row.
// W is read once and written once from HBM; T never leaves the CU.  Panels of
// all matrices of a batch are enumerated by one grid.
// ===========================================================================
template <int KT>
__global__ __launch_bounds__(256) void project_weights_mfma_bf16(PanelBatch pb,
                                                                 const uint16_t* __restrict__ U,
                                                                 int d, int k) {
  constexpr int KS2 = (KT + 1) / 2;
  constexpr int KPAD = 16 * KT;
  constexpr int LDK = 32 * KS2 + 4;       // LDS row pitch (floats) of T^T, padded
  constexpr int KW = (KT + 1) / 2;
  __shared__ float part[4][64 * LDK];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;

  int b = 0;
  const int blk = blockIdx.x;
  while (b + 1 < pb.count && blk >= pb.first_panel[b + 1]) ++b;
  uint16_t* __restrict__ W = pb.W[b];
  const int n = pb.n[b];
  const int j0 = (blk - pb.first_panel[b]) * 64;
  const bool full = (j0 + 64 <= n);
  const bool vec8 = full && (n % 4 == 0);
  const bool vec16 = full && (n % 8 == 0);
  const bool kfull = (k == KPAD);

  // ------------------------------ pass 1 ---------------------------------
  f32x4 acc[KT][4];
#pragma unroll
  for (int ti = 0; ti < KT; ++ti)
#pragma unroll
    for (int tj = 0; tj < 4; ++tj) acc[ti][tj] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nks = d >> 5;
  const int ucol0 = n16 * KT;
  const int wcol0 = j0 + 4 * n16;
  for (int s = wave; s < nks; s += 4) {
    const int row0 = 32 * s + 8 * g;
    uint32_t uw[8][KW], ww[8][2];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint16_t* up = U + (int64_t)(row0 + r) * k + ucol0;
      if (kfull && KT == 8) {
        u32x4 v = *(const u32x4*)up;
        uw[r][0] = v[0]; uw[r][1] = v[1]; uw[r][2] = v[2]; uw[r][3] = v[3];
      } else if (kfull && KT == 4) {
        u32x2 v = *(const u32x2*)up;
        uw[r][0] = v[0]; uw[r][1] = v[1];
      } else if (kfull && KT == 2) {
        uw[r][0] = *(const uint32_t*)up;
      } else {
#pragma unroll
        for (int w = 0; w < KW; ++w) {
          uint32_t lo = (ucol0 + 2 * w < k) ? (uint32_t)up[2 * w] : 0u;
          uint32_t hi = (2 * w + 1 < KT && ucol0 + 2 * w + 1 < k) ? (uint32_t)up[2 * w + 1] : 0u;
          uw[r][w] = lo | (hi << 16);
        }
      }
      const uint16_t* wp = W + (int64_t)(row0 + r) * n + wcol0;
      if (vec8) {
        u32x2 v = *(const u32x2*)wp;
        ww[r][0] = v[0]; ww[r][1] = v[1];
      } else {
        uint32_t e[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) e[c] = (wcol0 + c < n) ? (uint32_t)wp[c] : 0u;
        ww[r][0] = e[0] | (e[1] << 16);
        ww[r][1] = e[2] | (e[3] << 16);
      }
    }
    u32x4 ua[KT], wb[4];
#pragma unroll
    for (int i = 0; i < KT; ++i) {
      uint32_t f[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const uint32_t a = uw[2 * m][i >> 1], c = uw[2 * m + 1][i >> 1];
        f[m] = (i & 1) ? ((a >> 16) | (c & 0xFFFF0000u)) : ((a & 0xFFFFu) | (c << 16));
      }
      ua[i] = u32x4{f[0], f[1], f[2], f[3]};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t f[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const uint32_t a = ww[2 * m][i >> 1], c = ww[2 * m + 1][i >> 1];
        f[m] = (i & 1) ? ((a >> 16) | (c & 0xFFFF0000u)) : ((a & 0xFFFFu) | (c << 16));
      }
      wb[i] = u32x4{f[0], f[1], f[2], f[3]};
    }
#pragma unroll
    for (int ti = 0; ti < KT; ++ti)
#pragma unroll
      for (int tj = 0; tj < 4; ++tj) acc[ti][tj] = mfma16x16x32(ua[ti], wb[tj], acc[ti][tj]);
  }

  // partial T of this wave -> LDS, as T^T [j_local][kk]
  // lane (n16, g), element e of tile (ti, tj): kk = (4g+e)*KT + ti, j = 4*n16 + tj
  float* pw = part[wave];
#pragma unroll
  for (int tj = 0; tj < 4; ++tj)
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int ti = 0; ti < KT; ++ti)
        pw[(4 * n16 + tj) * LDK + (4 * g + e) * KT + ti] = acc[ti][tj][e];
  __syncthreads();
  for (int e = tid; e < 64 * LDK; e += 256) {
    const int kk = e % LDK;
    part[0][e] = (kk < KPAD) ? ((part[0][e] + part[1][e]) + (part[2][e] + part[3][e])) : 0.f;
  }
  __syncthreads();

  // ------------------------------ pass 2 ---------------------------------
  // A = T^T: row m <-> j_local = 16*(m/4) + 4*tj + m%4 ; K slots <-> kk = 32s+8g+0..7
  u32x4 thi[4][KS2], tlo[4][KS2];
  const int m4 = n16 >> 2, mr = n16 & 3;
#pragma unroll
  for (int tj = 0; tj < 4; ++tj)
#pragma unroll
    for (int s = 0; s < KS2; ++s) {
      const float* tp = &part[0][(16 * m4 + 4 * tj + mr) * LDK + 32 * s + 8 * g];
      f32x4 a = *(const f32x4*)tp;
      f32x4 c = *(const f32x4*)(tp + 4);
      float v[8] = {a[0], a[1], a[2], a[3], c[0], c[1], c[2], c[3]};
      split_bf16x8(v, thi[tj][s], tlo[tj][s]);
    }

  const int ndt = d >> 4;
  for (int dt = wave; dt < ndt; dt += 4) {
    const int drow = dt * 16 + n16;
    const uint16_t* up = U + (int64_t)drow * k + 8 * g;
    u32x4 ub[KS2];
#pragma unroll
    for (int s = 0; s < KS2; ++s)
      ub[s] = (32 * s + 8 * g < k) ? *(const u32x4*)(up + 32 * s) : u32x4{0u, 0u, 0u, 0u};
    f32x4 o[4];
#pragma unroll
    for (int tj = 0; tj < 4; ++tj) {
      f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS2; ++s) {
        a = mfma16x16x32(thi[tj][s], ub[s], a);
        a = mfma16x16x32(tlo[tj][s], ub[s], a);
      }
      o[tj] = a;
    }
    // lane holds W[drow][j0 + 16g + 4tj + e]
    uint16_t* wp = W + (int64_t)drow * n + j0 + 16 * g;
    if (vec16) {
      *(u32x4*)wp = u32x4{pack_bf16x2(o[0][0], o[0][1]), pack_bf16x2(o[0][2], o[0][3]),
                          pack_bf16x2(o[1][0], o[1][1]), pack_bf16x2(o[1][2], o[1][3])};
      *(u32x4*)(wp + 8) = u32x4{pack_bf16x2(o[2][0], o[2][1]), pack_bf16x2(o[2][2], o[2][3]),
                                pack_bf16x2(o[3][0], o[3][1]), pack_bf16x2(o[3][2], o[3][3])};
    } else {
#pragma unroll
      for (int tj = 0; tj < 4; ++tj)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (j0 + 16 * g + 4 * tj + e < n) wp[4 * tj + e] = (uint16_t)f32_to_bf16(o[tj][e]);
    }
  }
}

// ===========================================================================
// Column-partitioned kernel, bf16 storage, MFMA, every n a multiple of 8.
//
// The columns of all matrices of a batch form one sequence of 16-column
// tiles (a tile never spans two matrices).  Block b owns tiles
// [b*tpb, (b+1)*tpb), where tpb is chosen so that the grid is one block per
// compute unit: every block then streams the same number of bytes and the
// launch has no partial last round.  The block has tpb/2 waves (at least 4);
// wave w owns tiles w and w + waves for all k rows of T.
//   pass 1  T = U^T W over chunks of 64 rows.  The block loads each chunk of
//           W (a tile row is 32 contiguous bytes, the block's tiles of one
//           matrix are contiguous) and of U with 16-byte loads into a
//           row-major LDS tile; thread t moves piece t mod H of rows
//           t/H + 16i, so one pointer per thread serves every chunk.  Two
//           chunks are in flight in registers while one is computed.  The
//           waves read d-contiguous MFMA fragments of both tiles with LDS
//           transpose reads.
//   pass 2  W = U T over the same chunks: T^T is taken straight from each
//           wave's accumulators as bf16 hi + lo operand fragments, the U
//           chunk comes from LDS, and each wave writes its output tiles into
//           an LDS row tile that the whole block then stores with the same
//           contiguous 16-byte pattern it loaded W with (non-temporal: W is
//           not read again).
// W is read once and written once; U comes from L2 once per pass per block.
// ===========================================================================
struct ColumnBatch {
  uint16_t* W[kMaxBatch];
  int32_t n[kMaxBatch];
  int32_t first_tile[kMaxBatch + 1];   // prefix sums of ceil(n / 16)
  int32_t count;
  int32_t tiles;                       // total tiles of the batch
  int32_t tpb;                         // tiles per block
};

constexpr int kColRows = 64;           // rows per chunk
constexpr int kColMinWaves = 4;
// Waves per block at most: 10 (tiles per block <= 20) while the wave's
// registers allow three waves per SIMD; 8 for k > 64 or k % 8 != 0, and for
// three tiles per wave.
constexpr int cols_max_waves(int kt, bool kv, int ct) { return (kt > 4 || !kv || ct > 2) ? 8 : 10; }

// KV: k % 8 == 0, so U rows are whole 16-byte pieces.  Otherwise a chunk of
// U (64 whole rows, one contiguous span of 64*k bf16 that starts 16-byte
// aligned) is read with 16-byte loads and scattered element by element into
// the zero-padded row tile.
// NTL: W is read with non-temporal loads (each piece is read once and then
// overwritten by pass 2).  The 128-byte lines at the boundary of two strips
// are fetched by both blocks, and a streamed line is not kept for the
// neighbour.  Measured on MI355X (8-matrix batches, k = 64, d = 4096 and
// 5120, streamed against cached loads): 16 tiles per block (512-byte
// strips) 171 / 193 us, 18 tiles 204 / 233 us (d = 5120: 280 / 288), 20
// tiles 237 / 243 us; but 22 tiles 274 / 264 us, 23 tiles 452 / 413 us
// (d = 5120) and 361 / 320 us (d = 4096), and 9 tiles (288-byte strips,
// d = 2048) 85 / 78 us.  So the launcher streams for 16 to 20 tiles.
// XCD: blocks are dispatched to the 8 XCDs round robin (block b on XCD
// b mod 8); with XCD the block of launch index b takes strip
// (b mod 8) * (grid / 8) + b / 8, so that neighbouring strips, which share
// the 128-byte lines at their boundary, run on the same XCD and share its L2
// (needs grid % 8 == 0).
template <int KT, bool NTS, int DEPTH, bool KV, int CT = 2, bool NTL = false, bool XCD = false>
__global__ __launch_bounds__(kWave * cols_max_waves(KT, KV, CT)) void project_weights_cols_bf16(
    ColumnBatch cb, const uint16_t* __restrict__ U, int d, int k) {
  static_assert(DEPTH == 1 || DEPTH == 2, "one or two chunks in flight");
  static_assert(CT == 2 || CT == 3, "two or three tiles per wave");
  constexpr int R = kColRows;
  // rows per pass (threads t < RP*H each move one 16-byte piece per pass) and
  // W pieces per thread per chunk
  constexpr int RP = CT == 2 ? 16 : 8, NPW = R / RP;
  constexpr int KS2 = (KT + 1) / 2;
  constexpr int KW = 32 * KS2;                       // U tile width (bf16), zero padded past k
  constexpr int UPR = KW / 8;                        // U pieces (16 B) per row
  constexpr int UP = UPR + 1;                        // U row pitch in pieces
  constexpr int NUP = (R * UPR + kWave * kColMinWaves - 1) / (kWave * kColMinWaves);
  constexpr int WPMAX = 2 * CT * cols_max_waves(KT, KV, CT) + 1;
  __shared__ u32x4 wt[2][R * WPMAX];                 // W (pass 1) / output (pass 2) row tiles
  __shared__ u32x4 ut[2][R * UP];                    // U row tiles

  const int tid = threadIdx.x, NT = blockDim.x, NW = NT / kWave;
  const int lane = tid & 63, wave = tid >> 6;
  const int L = lane & 15, g = lane >> 4;
  const int tpb = cb.tpb;
  const int H = 2 * tpb, WP = H + 1;
  const int bx = XCD ? (int)((blockIdx.x % 8u) * (gridDim.x / 8u) + blockIdx.x / 8u) : (int)blockIdx.x;
  const int t0 = bx * tpb;
  const int tcount = min(tpb, cb.tiles - t0);
  const int nch = (d + R - 1) / R;

  // W pieces of this thread: piece h of rows row0 + RP*i of every chunk
  const bool wthr = tid < RP * H;
  const int h = tid % H, row0 = tid / H;
  int b = 0;
  {
    const int t = t0 + h / 2;
    while (b + 1 < cb.count && t >= cb.first_tile[b + 1]) ++b;
  }
  const int ld = cb.n[b];
  const int col = (t0 + h / 2 - cb.first_tile[b]) * 16 + 8 * (h & 1);
  const bool wok = wthr && h < 2 * tcount && col < ld;
  uint16_t* const wsrc = cb.W[b] + (int64_t)row0 * ld + col;
  const int wofs = row0 * WP + h;

  u32x4 wv[DEPTH][NPW], uv[DEPTH][NUP];
  auto load_w = [&](int c, u32x4 (&v)[NPW]) {
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int r = c * R + RP * i;
      const bool ok = wok && r + row0 < d;
      v[i] = ok ? ldg<NTL>(wsrc + (int64_t)r * ld) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto park_w = [&](int buf, const u32x4 (&v)[NPW]) {
    if (wthr)
#pragma unroll
      for (int i = 0; i < NPW; ++i) wt[buf][wofs + RP * i * WP] = v[i];
  };
  auto load_u = [&](int c, u32x4 (&v)[NUP]) {
#pragma unroll
    for (int i = 0; i < NUP; ++i) {
      const int q = tid + NT * i;
      if constexpr (KV) {
        const int r = c * R + q / UPR, uc = 8 * (q % UPR);
        const bool ok = q < R * UPR && uc < k && r < d;
        v[i] = ok ? *(const u32x4*)(U + (int64_t)r * k + uc) : u32x4{0u, 0u, 0u, 0u};
      } else {
        // piece q of the chunk's span; d % 32 == 0 makes the end of U fall on
        // a piece boundary
        const int64_t e0 = (int64_t)c * R * k + 8 * q;
        const bool ok = q < R * k / 8 && e0 + 8 <= (int64_t)d * k;
        v[i] = ok ? *(const u32x4*)(U + e0) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto park_u = [&](int buf, const u32x4 (&v)[NUP]) {
#pragma unroll
    for (int i = 0; i < NUP; ++i) {
      const int q = tid + NT * i;
      if constexpr (KV) {
        if (q < R * UPR) ut[buf][(q / UPR) * UP + q % UPR] = v[i];
      } else if (q < R * k / 8) {
        uint16_t* t = (uint16_t*)ut[buf];
        int r = (8 * q) / k, col = 8 * q - r * k;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t w = v[i][e >> 1];
          t[r * (8 * UP) + col] = (uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu));
          if (++col == k) {
            col = 0;
            ++r;
          }
        }
      }
    }
  };
  if constexpr (!KV) {
    // columns k .. KW of the U tiles are never written by the scatter
    for (int i = tid; i < 2 * R * UP; i += NT) (&ut[0][0])[i] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
  }

  // ------------------------------ pass 1 ---------------------------------
  f32x4 acc[KT][CT];
#pragma unroll
  for (int i = 0; i < KT; ++i)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute1 = [&](int c) {
    const uint16_t* ub = (const uint16_t*)ut[c & 1];
    const uint16_t* wb = (const uint16_t*)wt[c & 1];
#pragma unroll
    for (int ks = 0; ks < R / 32; ++ks) {
      const int r = 32 * ks + 8 * g + (L >> 2);
      u32x4 a[KT];
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        const uint16_t* p = ub + r * (8 * UP) + 16 * i + 4 * (L & 3);
        const u32x2 x = lds_read_tr16(p), y = lds_read_tr16(p + 4 * 8 * UP);
        a[i] = u32x4{x[0], x[1], y[0], y[1]};
      }
#pragma unroll
      for (int cc = 0; cc < CT; ++cc) {
        const int jl = wave + NW * cc;
        if (jl < tcount) {
          const uint16_t* p = wb + r * (8 * WP) + 16 * jl + 4 * (L & 3);
          const u32x2 x = lds_read_tr16(p), y = lds_read_tr16(p + 4 * 8 * WP);
          const u32x4 bfr = u32x4{x[0], x[1], y[0], y[1]};
#pragma unroll
          for (int i = 0; i < KT; ++i) acc[i][cc] = mfma16x16x32(a[i], bfr, acc[i][cc]);
        }
      }
    }
  };
  // chunk 0 parked, chunks 1 .. DEPTH in flight; chunk j travels in set j % DEPTH
  load_w(0, wv[0]);
  load_u(0, uv[0]);
  park_w(0, wv[0]);
  park_u(0, uv[0]);
#pragma unroll
  for (int j = 1; j <= DEPTH; ++j)
    if (j < nch) {
      load_w(j, wv[j % DEPTH]);
      load_u(j, uv[j % DEPTH]);
    }
  __syncthreads();
  auto step1 = [&](int c, auto S) {
    constexpr int s = decltype(S)::value;      // == (c + 1) % DEPTH
    compute1(c);
    if (c + 1 < nch) {
      park_w((c + 1) & 1, wv[s]);
      park_u((c + 1) & 1, uv[s]);
    }
    if (c + 1 + DEPTH < nch) {
      load_w(c + 1 + DEPTH, wv[s]);
      load_u(c + 1 + DEPTH, uv[s]);
    }
    __syncthreads();
  };
  for (int c = 0; c < nch; c += DEPTH) {
    step1(c, std::integral_constant<int, 1 % DEPTH>{});
    if constexpr (DEPTH == 2)
      if (c + 1 < nch) step1(c + 1, std::integral_constant<int, 0>{});
  }

  // ------------------------------ pass 2 ---------------------------------
  // A = T^T: row m <-> column 16*jl + m; K slot (g, r) <-> k index
  // 32s + 4g + r (r < 4) or 32s + 16 + 4g + r - 4 (r >= 4), which is exactly
  // what acc[2s][cc] and acc[2s+1][cc] of this lane hold.
  u32x4 thi[CT][KS2], tlo[CT][KS2];
#pragma unroll
  for (int cc = 0; cc < CT; ++cc)
#pragma unroll
    for (int s = 0; s < KS2; ++s) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = acc[2 * s][cc][e];
        v[4 + e] = (2 * s + 1 < KT) ? acc[2 * s + 1][cc][e] : 0.f;
      }
      split_bf16x8(v, thi[cc][s], tlo[cc][s]);
    }

  load_u(0, uv[0]);
  park_u(0, uv[0]);
  if (nch > 1) load_u(1, uv[0]);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const uint16_t* ub = (const uint16_t*)ut[c & 1];
    uint16_t* ob = (uint16_t*)wt[c & 1];
#pragma unroll
    for (int sub = 0; sub < R / 16; ++sub) {
      const int r = 16 * sub + L;
      u32x4 bfr[KS2];
#pragma unroll
      for (int s = 0; s < KS2; ++s) {
        const uint16_t* p = ub + r * (8 * UP) + 32 * s + 4 * g;
        const u32x2 x = *(const u32x2*)p, y = *(const u32x2*)(p + 16);
        bfr[s] = u32x4{x[0], x[1], y[0], y[1]};
      }
#pragma unroll
      for (int cc = 0; cc < CT; ++cc) {
        const int jl = wave + NW * cc;
        if (jl < tcount) {
          f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < KS2; ++s) {
            o = mfma16x16x32(thi[cc][s], bfr[s], o);
            o = mfma16x16x32(tlo[cc][s], bfr[s], o);
          }
          // lane holds W[row r of the chunk][16*jl + 4g + 0..3]
          *(u32x2*)(ob + r * (8 * WP) + 16 * jl + 4 * g) =
              u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
        }
      }
    }
    if (c + 1 < nch) park_u((c + 1) & 1, uv[0]);
    if (c + 2 < nch) load_u(c + 2, uv[0]);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int r = c * R + RP * i;
      if (wok && r + row0 < d) stg<NTS>(wsrc + (int64_t)r * ld, wt[c & 1][wofs + RP * i * WP]);
    }
  }
}

// ===========================================================================
// Generic kernel: any dtype, d, k <= 1024.  One block per column (grid-
// stride): t = U^T w by block reductions in fixed order, then w <- U t.
// ===========================================================================
constexpr int kGenericMaxK = 1024;

template <typename T>
__global__ __launch_bounds__(256) void project_weights_generic(T* __restrict__ W,
                                                               const T* __restrict__ U,
                                                               int64_t d, int64_t n, int64_t k) {
  __shared__ float tcol[kGenericMaxK];
  __shared__ float red[8][256];
  const int tid = threadIdx.x;
  for (int64_t j = blockIdx.x; j < n; j += gridDim.x) {
    for (int64_t kc = 0; kc < k; kc += 8) {
      float p[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] = 0.f;
      for (int64_t r = tid; r < d; r += 256) {
        const float w = load_as_f32(W + r * n + j);
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (kc + i < k) p[i] = fmaf(load_as_f32(U + r * k + kc + i), w, p[i]);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) red[i][tid] = p[i];
      __syncthreads();
      for (int h = 128; h >= 1; h >>= 1) {
        if (tid < h)
#pragma unroll
          for (int i = 0; i < 8; ++i) red[i][tid] += red[i][tid + h];
        __syncthreads();
      }
      if (tid < 8 && kc + tid < k) tcol[kc + tid] = red[tid][0];
      __syncthreads();
    }
    for (int64_t r = tid; r < d; r += 256) {
      float a = 0.f;
      for (int64_t c = 0; c < k; ++c) a = fmaf(load_as_f32(U + r * k + c), tcol[c], a);
      store_from_f32(W + r * n + j, a);
    }
    __syncthreads();
  }
}

bool weights_use_mfma(int dtype, int64_t d, int64_t k) {
  return dtype == kBF16 && d % 32 == 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

template <int KT>
static hipError_t launch_weights_kt(const PanelBatch& pb, int blocks, const void* U, int d, int k,
                                    hipStream_t st) {
  hipLaunchKernelGGL((project_weights_mfma_bf16<KT>), dim3(blocks), dim3(256), 0, st, pb,
                     (const uint16_t*)U, d, k);
  return hipGetLastError();
}

// Cached per device; calls from several host threads may fill an entry
// concurrently, each with the same value (relaxed atomics).
int device_cu_count() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0)
      c = 256;
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

template <int KT, bool KV>
static hipError_t launch_cols_kv(ColumnBatch cb, int cus, const void* U, int d, int k, hipStream_t st) {
  // one chunk in flight where two would spill registers (k > 64, k % 8 != 0)
  constexpr int DEPTH = (KT > 4 && !KV) ? 1 : 2;
  constexpr int W2 = cols_max_waves(KT, KV, 2), W3 = cols_max_waves(KT, KV, 3);
  // three tiles per wave only for k <= 64, where its registers fit
  constexpr int kMaxTpb = KT <= 4 ? 3 * W3 : 2 * W2;
  int tpb = (cb.tiles + cus - 1) / cus;
  cb.tpb = tpb < 1 ? 1 : (tpb > kMaxTpb ? kMaxTpb : tpb);
  const unsigned grid = (unsigned)((cb.tiles + cb.tpb - 1) / cb.tpb);
  // XCD-aware strip order when the grid is a multiple of the 8 XCDs;
  // streamed W loads with k % 8 == 0 and 16 to 20 tiles per block (measured)
  const bool xcd = grid % 8 == 0;
  const bool ntl = KV && cb.tpb >= 16 && cb.tpb <= 20;
#define SSN_COLS(CT)                                                                              \
  do {                                                                                            \
    if (xcd && ntl)                                                                               \
      hipLaunchKernelGGL((project_weights_cols_bf16<KT, true, DEPTH, KV, CT, true, true>), dim3(grid), \
                         dim3(kWave * waves), 0, st, cb, (const uint16_t*)U, d, k);               \
    else if (xcd)                                                                                 \
      hipLaunchKernelGGL((project_weights_cols_bf16<KT, true, DEPTH, KV, CT, false, true>), dim3(grid), \
                         dim3(kWave * waves), 0, st, cb, (const uint16_t*)U, d, k);               \
    else                                                                                          \
      hipLaunchKernelGGL((project_weights_cols_bf16<KT, true, DEPTH, KV, CT, false, false>), dim3(grid), \
                         dim3(kWave * waves), 0, st, cb, (const uint16_t*)U, d, k);               \
  } while (0)
  if (cb.tpb <= 2 * W2) {
    int waves = (cb.tpb + 1) / 2;
    waves = waves < kColMinWaves ? kColMinWaves : waves;
    SSN_COLS(2);
  } else if constexpr (KT <= 4) {
    const int waves = (cb.tpb + 2) / 3;
    SSN_COLS(3);
  }
#undef SSN_COLS
  return hipGetLastError();
}

template <int KT>
static hipError_t launch_cols(const ColumnBatch& cb, int cus, const void* U, int d, int k, hipStream_t st) {
  return k % 8 == 0 ? launch_cols_kv<KT, true>(cb, cus, U, d, k, st)
                    : launch_cols_kv<KT, false>(cb, cus, U, d, k, st);
}

hipError_t launch_project_weights(int dtype, int count, int64_t d, const int64_t* n, int64_t k,
                                  void* const* W, const void* U, hipStream_t st) {
  bool aligned = (((uintptr_t)U & 15u) == 0);
  bool cols8 = true, cols4 = true;
  // the MFMA kernels keep each matrix's row stride n in 32 bits; wider
  // matrices take the generic kernel, whose indexing is 64-bit throughout
  bool n32 = true;
  int64_t panels = 0, tiles = 0;
  for (int b = 0; b < count; ++b) {
    aligned = aligned && (((uintptr_t)W[b] & 15u) == 0);
    cols8 = cols8 && (n[b] % 8 == 0);
    cols4 = cols4 && (n[b] % 4 == 0);
    n32 = n32 && n[b] <= INT32_MAX;
    panels += (n[b] + 63) / 64;
    tiles += (n[b] + 15) / 16;
  }
  if (dtype == kF32 && weights_f32_uses_mfma(d, k) && aligned && n32 && cols4 && tiles <= INT32_MAX / 2) {
    float* Wf[kMaxBatch];
    for (int b = 0; b < count; ++b) Wf[b] = (float*)W[b];
    return launch_project_weights_f32(count, d, n, k, Wf, (const float*)U, st);
  }
  const bool mfma = weights_use_mfma(dtype, d, k) && aligned && n32;
  if (mfma && cols8 && tiles <= INT32_MAX / 2) {
    ColumnBatch cb{};
    int nb = 0;
    int32_t acc = 0;
    for (int b = 0; b < count; ++b) {
      if (n[b] == 0) continue;
      cb.W[nb] = (uint16_t*)W[b];
      cb.n[nb] = (int32_t)n[b];
      cb.first_tile[nb] = acc;
      acc += (int32_t)((n[b] + 15) / 16);
      ++nb;
    }
    if (nb == 0) return hipSuccess;
    for (int b = nb; b <= kMaxBatch; ++b) cb.first_tile[b] = acc;
    cb.count = nb;
    cb.tiles = acc;
    const int cus = device_cu_count();
    const int kt = (int)((k + 15) / 16);
    if (kt <= 2) return launch_cols<2>(cb, cus, U, (int)d, (int)k, st);
    if (kt <= 4) return launch_cols<4>(cb, cus, U, (int)d, (int)k, st);
    return launch_cols<8>(cb, cus, U, (int)d, (int)k, st);
  }
  // the 64-column panel kernel reads U rows as 16-byte pieces: k % 8 == 0
  if (mfma && k % 8 == 0 && panels <= INT32_MAX) {
    PanelBatch pb{};
    int nb = 0;
    int32_t acc = 0;
    for (int b = 0; b < count; ++b) {
      if (n[b] == 0) continue;
      pb.W[nb] = (uint16_t*)W[b];
      pb.n[nb] = (int32_t)n[b];
      pb.first_panel[nb] = acc;
      acc += (int32_t)((n[b] + 63) / 64);
      ++nb;
    }
    pb.first_panel[nb] = acc;
    pb.count = nb;
    if (nb == 0) return hipSuccess;
    switch ((k + 15) / 16) {
      case 1: return launch_weights_kt<1>(pb, acc, U, (int)d, (int)k, st);
      case 2: return launch_weights_kt<2>(pb, acc, U, (int)d, (int)k, st);
      case 3: return launch_weights_kt<3>(pb, acc, U, (int)d, (int)k, st);
      case 4: return launch_weights_kt<4>(pb, acc, U, (int)d, (int)k, st);
      case 5: return launch_weights_kt<5>(pb, acc, U, (int)d, (int)k, st);
      case 6: return launch_weights_kt<6>(pb, acc, U, (int)d, (int)k, st);
      case 7: return launch_weights_kt<7>(pb, acc, U, (int)d, (int)k, st);
      default: return launch_weights_kt<8>(pb, acc, U, (int)d, (int)k, st);
    }
  }
  for (int b = 0; b < count; ++b) {
    if (n[b] == 0) continue;
    const unsigned grid = (unsigned)(n[b] < 65536 ? n[b] : 65536);
    if (dtype == kF32)
      hipLaunchKernelGGL((project_weights_generic<float>), dim3(grid), dim3(256), 0, st,
                         (float*)W[b], (const float*)U, d, n[b], k);
    else
      hipLaunchKernelGGL((project_weights_generic<uint16_t>), dim3(grid), dim3(256), 0, st,
                         (uint16_t*)W[b], (const uint16_t*)U, d, n[b], k);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ssn

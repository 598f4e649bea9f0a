// Stage-boundary codec kernels: compress / gradient projection (contract over
// d) and decompress / gradient expansion (contract over k).
//
// Paper: section 4.1, Eq. (2) -- Z = (X - E[ids]) U, reconstruction with U^T,
// and "the backward pass uses the same compression" (G_Z = G U at the
// receiver, G_Z U^T at the sender).
#include "ssn_device.h"
#include "ssn_launch.h"

namespace ssn {

// ===========================================================================
// compress / project_grad, bf16 storage, MFMA 16x16x32 with fp32 accumulate.
//
// Block = 4 waves; wave w owns 16*MT consecutive tokens (one MFMA M tile per
// 16 tokens).  d is walked in chunks of DC = 32*KS.  For every chunk the 256
// threads stage that slice of U into LDS already in B-fragment order (double
// buffered, one barrier per chunk); X and E[ids] rows go from HBM straight into
// A-fragment registers with 16-byte loads, one chunk ahead of the MFMAs.
//
// B-fragment construction (U is [d][k], k contiguous; a fragment needs 8
// consecutive d for one column): lane position n of K-group g loads the
// 8 x KP block U[d0+8g .. +7][n*KP .. n*KP+KP-1] and transposes it in
// registers into KP fragments; fragment i carries column n*KP + i.  MFMA N
// tile i therefore produces columns {n*KP + i}, so after the KP tiles each
// lane holds KP consecutive columns of Z per token: contiguous stores.
//
// The embedding subtraction is fused by linearity: X.U and E[ids].U are
// accumulated by identical MFMA sequences into separate fp32 accumulators
// and subtracted once at the end (compress(E[ids]) is exactly zero).
// ===========================================================================
template <int KP, int MT, int KS, bool HAS_E>
__global__ __launch_bounds__(256) void compress_mfma_bf16(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    float* __restrict__ Z, int64_t N, int d, int k, int64_t V) {
  constexpr int DC = 32 * KS;
  constexpr int FRAGS = KS * KP * kWave;          // u32x4 fragments per LDS buffer
  constexpr int TASKS = KS * kWave;               // staging tasks per chunk
  constexpr int TPT = (TASKS + 255) / 256;        // tasks per thread
  constexpr int KW = (KP + 1) / 2;                // dwords per staged row
  __shared__ u32x4 lds[2][FRAGS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * MT);
  const bool kfull = (k == 16 * KP);

  const uint16_t* xrow[MT];
  const uint16_t* erow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int64_t t = tok0 + mt * 16 + n16;
    t = t < N ? t : N - 1;
    xrow[mt] = X + t * d + 8 * g;
    if (HAS_E) erow[mt] = E + clamp_id(ids[t], V) * d + 8 * g;
  }

  const int nchunks = (d + DC - 1) / DC;

  // ---- U staging: global -> registers (8 rows x KP columns per task) ----
  uint32_t st[TPT][8][KW];
  auto stage_load = [&](int c) {
#pragma unroll
    for (int q = 0; q < TPT; ++q) {
      const int t = tid + 256 * q;
      const int s = t >> 6, l = t & 63;
      const int row0 = c * DC + 32 * s + 8 * (l >> 4);
      const int col0 = (l & 15) * KP;
      if (t < TASKS && row0 < d) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const uint16_t* p = U + (int64_t)(row0 + r) * k + col0;
          if (kfull && KP == 8) {
            u32x4 v = *(const u32x4*)p;
            st[q][r][0] = v[0]; st[q][r][1] = v[1]; st[q][r][2] = v[2]; st[q][r][3] = v[3];
          } else if (kfull && KP == 4) {
            u32x2 v = *(const u32x2*)p;
            st[q][r][0] = v[0]; st[q][r][1] = v[1];
          } else if (kfull && (KP % 2) == 0) {
#pragma unroll
            for (int w = 0; w < KW; ++w) st[q][r][w] = ((const uint32_t*)p)[w];
          } else {
#pragma unroll
            for (int w = 0; w < KW; ++w) {
              uint32_t lo = (col0 + 2 * w < k) ? (uint32_t)p[2 * w] : 0u;
              uint32_t hi = (2 * w + 1 < KP && col0 + 2 * w + 1 < k) ? (uint32_t)p[2 * w + 1] : 0u;
              st[q][r][w] = lo | (hi << 16);
            }
          }
        }
      }
    }
  };
  // ---- registers -> LDS in B-fragment order (8x2 transposes) ----
  auto stage_store = [&](int buf, int c) {
#pragma unroll
    for (int q = 0; q < TPT; ++q) {
      const int t = tid + 256 * q;
      const int s = t >> 6, l = t & 63;
      const int row0 = c * DC + 32 * s + 8 * (l >> 4);
      if (t < TASKS && row0 < d) {
#pragma unroll
        for (int i = 0; i < KP; ++i) {
          uint32_t f[4];
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            const uint32_t a = st[q][2 * m][i >> 1], b = st[q][2 * m + 1][i >> 1];
            f[m] = (i & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
          }
          lds[buf][(s * KP + i) * kWave + l] = u32x4{f[0], f[1], f[2], f[3]};
        }
      }
    }
  };

  u32x4 xa[MT][KS], ea[MT][KS];
  auto load_frags = [&](int c, u32x4 (&xo)[MT][KS], u32x4 (&eo)[MT][KS]) {
    const int kv = min(KS, (d - c * DC) >> 5);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int s = 0; s < KS; ++s)
        if (s < kv) {
          xo[mt][s] = *(const u32x4*)(xrow[mt] + c * DC + 32 * s);
          if (HAS_E) eo[mt][s] = *(const u32x4*)(erow[mt] + c * DC + 32 * s);
        }
  };

  f32x4 accX[MT][KP], accE[MT][KP];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int i = 0; i < KP; ++i) {
      accX[mt][i] = f32x4{0.f, 0.f, 0.f, 0.f};
      accE[mt][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

  load_frags(0, xa, ea);
  stage_load(0);
  stage_store(0, 0);

  for (int c = 0; c < nchunks; ++c) {
    const int kv = min(KS, (d - c * DC) >> 5);
    const bool more = (c + 1 < nchunks);
    u32x4 xn[MT][KS], en[MT][KS];
    if (more) {
      load_frags(c + 1, xn, en);
      stage_load(c + 1);
    }
    __syncthreads();
    const u32x4* fr = lds[c & 1];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (s < kv) {
        u32x4 b[KP];
#pragma unroll
        for (int i = 0; i < KP; ++i) b[i] = fr[(s * KP + i) * kWave + lane];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int i = 0; i < KP; ++i) {
            accX[mt][i] = mfma16x16x32(xa[mt][s], b[i], accX[mt][i]);
            if (HAS_E) accE[mt][i] = mfma16x16x32(ea[mt][s], b[i], accE[mt][i]);
          }
      }
    }
    if (more) {
      stage_store((c + 1) & 1, c + 1);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          xa[mt][s] = xn[mt][s];
          if (HAS_E) ea[mt][s] = en[mt][s];
        }
    }
  }

  // ---- epilogue: lane (n16, g) holds Z[tok0+16mt+4g+j][n16*KP + i] ----
  const int col0 = n16 * KP;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t t = tok0 + mt * 16 + 4 * g + j;
      if (t < N) {
        float v[KP];
#pragma unroll
        for (int i = 0; i < KP; ++i) v[i] = HAS_E ? accX[mt][i][j] - accE[mt][i][j] : accX[mt][i][j];
        float* zp = Z + t * k + col0;
        if (kfull && KP % 4 == 0) {
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
// so that U is used in its natural [d][k] layout (A fragment = 16 contiguous
// bytes of one U row) and Z rows are B fragments.  Z (fp32) is split into bf16
// hi + lo parts, two MFMAs each, which keeps ~fp32 accuracy.  The accumulator
// starts from E[ids] (widened to fp32) -- the embedding add is fused and the
// result is rounded to bf16 once.
//
// Block = 4 waves sharing 16*TG tokens; the waves split d in steps of 64.  A
// 64-wide d step uses 4 MFMA tiles whose rows are permuted so that each lane
// ends with 16 consecutive d of one token: 32-byte E loads and Y stores.
// ===========================================================================
template <int KS2, int TG, bool HAS_E>
__global__ __launch_bounds__(256) void decompress_mfma_bf16(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    uint16_t* __restrict__ Y, int64_t N, int d, int k, int64_t V) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tokb = (int64_t)blockIdx.x * (16 * TG);

  // Z^T B fragments (hi/lo) for the block's tokens.
  u32x4 zhi[TG][KS2], zlo[TG][KS2];
  const uint16_t* erow[TG];
  uint16_t* yrow[TG];
  bool tok_ok[TG];
#pragma unroll
  for (int tg = 0; tg < TG; ++tg) {
    int64_t t = tokb + tg * 16 + n16;
    tok_ok[tg] = t < N;
    t = t < N ? t : N - 1;
    yrow[tg] = Y + t * d + 16 * g;
    if (HAS_E) erow[tg] = E + clamp_id(ids[t], V) * d + 16 * g;
    const float* zp = Zc + t * k;
#pragma unroll
    for (int s = 0; s < KS2; ++s) {
      const int c0 = 32 * s + 8 * g;
      float v[8];
      if (c0 + 8 <= k) {
        f32x4 a = *(const f32x4*)(zp + c0);
        f32x4 b = *(const f32x4*)(zp + c0 + 4);
        v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
        v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;   // k % 8 == 0 on this path
      }
      split_bf16x8(v, zhi[tg][s], zlo[tg][s]);
    }
  }

  const int m4 = n16 >> 2, mr = n16 & 3;
  const int nsteps = d >> 6;
  for (int ds = wave; ds < nsteps; ds += 4) {
    const int dbase = ds * 64;
    // A fragments: tile t row n16 <-> d = dbase + 16*(n16/4) + 4t + n16%4
    u32x4 ua[4][KS2];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint16_t* up = U + (int64_t)(dbase + 16 * m4 + 4 * t + mr) * k + 8 * g;
#pragma unroll
      for (int s = 0; s < KS2; ++s)
        ua[t][s] = (32 * s + 8 * g < k) ? *(const u32x4*)(up + 32 * s) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int tg = 0; tg < TG; ++tg) {
      f32x4 acc[4];
      if (HAS_E) {
        u32x4 e0 = *(const u32x4*)(erow[tg] + dbase);
        u32x4 e1 = *(const u32x4*)(erow[tg] + dbase + 8);
        acc[0] = f32x4{lo_bf16(e0[0]), hi_bf16(e0[0]), lo_bf16(e0[1]), hi_bf16(e0[1])};
        acc[1] = f32x4{lo_bf16(e0[2]), hi_bf16(e0[2]), lo_bf16(e0[3]), hi_bf16(e0[3])};
        acc[2] = f32x4{lo_bf16(e1[0]), hi_bf16(e1[0]), lo_bf16(e1[1]), hi_bf16(e1[1])};
        acc[3] = f32x4{lo_bf16(e1[2]), hi_bf16(e1[2]), lo_bf16(e1[3]), hi_bf16(e1[3])};
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int s = 0; s < KS2; ++s) {
          acc[t] = mfma16x16x32(ua[t][s], zhi[tg][s], acc[t]);
          acc[t] = mfma16x16x32(ua[t][s], zlo[tg][s], acc[t]);
        }
      if (tok_ok[tg]) {
        u32x4 o0 = u32x4{pack_bf16x2(acc[0][0], acc[0][1]), pack_bf16x2(acc[0][2], acc[0][3]),
                         pack_bf16x2(acc[1][0], acc[1][1]), pack_bf16x2(acc[1][2], acc[1][3])};
        u32x4 o1 = u32x4{pack_bf16x2(acc[2][0], acc[2][1]), pack_bf16x2(acc[2][2], acc[2][3]),
                         pack_bf16x2(acc[3][0], acc[3][1]), pack_bf16x2(acc[3][2], acc[3][3])};
        *(u32x4*)(yrow[tg] + dbase) = o0;
        *(u32x4*)(yrow[tg] + dbase + 8) = o1;
      }
    }
  }
}

// ===========================================================================
// Generic kernels: any storage dtype, any d and k.  One wave per token,
// fp32 arithmetic, wavefront reductions.  Used for fp32 storage and for shapes
// the MFMA kernels do not tile.
// ===========================================================================
template <typename T, bool HAS_E>
__global__ __launch_bounds__(256) void compress_generic(
    const T* __restrict__ X, const int32_t* __restrict__ ids, const T* __restrict__ E,
    const T* __restrict__ U, float* __restrict__ Z, int64_t N, int64_t d, int64_t k, int64_t V) {
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
      if (lane < 16 && kc + lane < k) Z[t * k + kc + lane] = mine;
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
  return dtype == kBF16 && d % 32 == 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

bool decompress_uses_mfma(int dtype, int64_t d, int64_t k) {
  return dtype == kBF16 && d % 64 == 0 && d <= INT32_MAX && k % 8 == 0 && k >= 8 && k <= 128;
}

template <int KP, bool HAS_E>
static hipError_t launch_compress_kp(int64_t N, int d, int k, int64_t V, const void* X,
                                     const int32_t* ids, const void* E, const void* U, float* Z,
                                     hipStream_t st) {
  constexpr int MT = 1;
  constexpr int KS = (KP > 4) ? 2 : 4;
  const int64_t per_block = 4 * 16 * MT;
  const int64_t blocks = (N + per_block - 1) / per_block;
  hipLaunchKernelGGL((compress_mfma_bf16<KP, MT, KS, HAS_E>), dim3((unsigned)blocks), dim3(256), 0,
                     st, (const uint16_t*)X, ids, (const uint16_t*)E, (const uint16_t*)U, Z, N, d,
                     k, V);
  return hipGetLastError();
}

template <bool HAS_E>
static hipError_t launch_compress_mfma(int64_t N, int d, int k, int64_t V, const void* X,
                                       const int32_t* ids, const void* E, const void* U, float* Z,
                                       hipStream_t st) {
  switch ((k + 15) / 16) {
    case 1: return launch_compress_kp<1, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    case 2: return launch_compress_kp<2, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    case 3: return launch_compress_kp<3, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    case 4: return launch_compress_kp<4, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    case 5: return launch_compress_kp<5, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    case 6: return launch_compress_kp<6, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    case 7: return launch_compress_kp<7, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
    default: return launch_compress_kp<8, HAS_E>(N, d, k, V, X, ids, E, U, Z, st);
  }
}

static unsigned generic_blocks(int64_t N) {
  const int64_t want = (N + 3) / 4;
  return (unsigned)(want < 65536 ? want : 65536);
}

hipError_t launch_compress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const void* X,
                           const int32_t* ids, const void* E, const void* U, float* Z,
                           hipStream_t st) {
  const bool has_e = (E != nullptr);
  if (compress_uses_mfma(dtype, d, k) && al16(X) && al16(U) && al16(Z) && (!has_e || al16(E))) {
    return has_e ? launch_compress_mfma<true>(N, (int)d, (int)k, V, X, ids, E, U, Z, st)
                 : launch_compress_mfma<false>(N, (int)d, (int)k, V, X, ids, E, U, Z, st);
  }
  const unsigned nb = generic_blocks(N);
  if (dtype == kF32) {
    if (has_e)
      hipLaunchKernelGGL((compress_generic<float, true>), dim3(nb), dim3(256), 0, st,
                         (const float*)X, ids, (const float*)E, (const float*)U, Z, N, d, k, V);
    else
      hipLaunchKernelGGL((compress_generic<float, false>), dim3(nb), dim3(256), 0, st,
                         (const float*)X, ids, (const float*)E, (const float*)U, Z, N, d, k, V);
  } else {
    if (has_e)
      hipLaunchKernelGGL((compress_generic<uint16_t, true>), dim3(nb), dim3(256), 0, st,
                         (const uint16_t*)X, ids, (const uint16_t*)E, (const uint16_t*)U, Z, N, d,
                         k, V);
    else
      hipLaunchKernelGGL((compress_generic<uint16_t, false>), dim3(nb), dim3(256), 0, st,
                         (const uint16_t*)X, ids, (const uint16_t*)E, (const uint16_t*)U, Z, N, d,
                         k, V);
  }
  return hipGetLastError();
}

template <int KS2, bool HAS_E>
static hipError_t launch_decompress_ks(int64_t N, int d, int k, int64_t V, const float* Zc,
                                       const int32_t* ids, const void* E, const void* U, void* Y,
                                       hipStream_t st) {
  constexpr int TG = (KS2 > 2) ? 2 : 4;
  const int64_t per_block = 16 * TG;
  const int64_t blocks = (N + per_block - 1) / per_block;
  hipLaunchKernelGGL((decompress_mfma_bf16<KS2, TG, HAS_E>), dim3((unsigned)blocks), dim3(256), 0,
                     st, Zc, ids, (const uint16_t*)E, (const uint16_t*)U, (uint16_t*)Y, N, d, k, V);
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

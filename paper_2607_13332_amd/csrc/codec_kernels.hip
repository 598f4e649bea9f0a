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
constexpr int kCompressKS = 4;                 // K steps (of 32) per d chunk
constexpr int kCompressDC = 32 * kCompressKS;  // d chunk

template <int KP, int NBUF, bool HAS_E, bool KFULL, bool ROT = false, bool NT = false,
          int WAVES = 4, int KS = kCompressKS>
__global__ __launch_bounds__(64 * WAVES) void compress_mfma_bf16(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    float* __restrict__ Z, int64_t N, int d, int k, int64_t V) {
  constexpr int DC = 32 * KS;
  constexpr int KW = (KP + 1) / 2;
  constexpr int TASKS = KS * kWave;            // staging tasks per chunk
  static_assert(TASKS % (64 * WAVES) == 0 || (64 * WAVES) % TASKS == 0, "staging split");
  constexpr int TPT = TASKS >= 64 * WAVES ? TASKS / (64 * WAVES) : 1;
  __shared__ u32x4 lds[2][KS * KP * kWave];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tok0 = ((int64_t)blockIdx.x * WAVES + wave) * 16;
  int64_t t = tok0 + n16;
  t = t < N ? t : N - 1;
  const uint16_t* xrow = X + t * d + 8 * g;
  const uint16_t* erow = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * g : nullptr;

  // staging tasks of this thread: task t = tid + q*64*WAVES covers K step
  // t/64, K group (t/16)%4, column block t%16 of the chunk
  const bool stager = tid < TASKS;
  int srow[TPT], sidx[TPT];
#pragma unroll
  for (int q = 0; q < TPT; ++q) {
    const int t = tid + q * 64 * WAVES;
    srow[q] = 32 * (t >> 6) + 8 * ((t >> 4) & 3);
    sidx[q] = (t >> 6) * KP * kWave + (t & 63);
  }
  const int scol = (tid & 15) * KP;
  const int nch = d / DC;
  // Each block sweeps the d chunks starting at its own offset: if every wave
  // read the same column range of its rows at the same time, the requests
  // would pile onto a few HBM channels.
  const int rot = ROT ? (int)(blockIdx.x % (unsigned)nch) : 0;
  auto chunk = [&](int c) { const int x = c + rot; return x < nch ? x : x - nch; };

  u32x4 xf[NBUF][KS], ef[NBUF][KS];
  uint32_t uw[TPT][8][KW];

  auto load_xe = [&](int c, u32x4(&xo)[KS], u32x4(&eo)[KS]) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      xo[s] = ldg<NT>(xrow + c * DC + 32 * s);
      if constexpr (HAS_E) eo[s] = ldg<NT>(erow + c * DC + 32 * s);
    }
  };
  auto load_u = [&](int c) {
    if (stager) {
#pragma unroll
      for (int q = 0; q < TPT; ++q)
        load_block8<KP, KFULL>(U, (int64_t)c * DC + srow[q], scol, k, k, uw[q]);
    }
  };
  auto store_u = [&](int buf) {
    if (stager) {
#pragma unroll
      for (int q = 0; q < TPT; ++q)
#pragma unroll
        for (int i = 0; i < KP; ++i) lds[buf][sidx[q] + i * kWave] = block8_column<KP>(uw[q], i);
    }
  };

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
// so that U is used in its natural [d][k] layout (A fragment = 16 contiguous
// bytes of one U row) and Z rows are B fragments.  Z (fp32) is split into bf16
// hi + lo parts, two MFMAs each, which keeps ~fp32 accuracy.  The accumulator
// starts from E[ids] (widened to fp32) -- the embedding add is fused and the
// result is rounded to bf16 once.
//
// Block = 4 waves sharing 16*TG tokens; the waves split d in steps of 64
// (wave w takes steps w, w+4, ...).  A 64-wide d step uses 4 MFMA tiles whose
// rows are permuted so that lane (token n, group g) ends with d offsets
// 8g..8g+7 (tiles 0, 1) and 32+8g..32+8g+7 (tiles 2, 3) of one token: each
// E load and Y store instruction then covers 64 contiguous bytes of 16 rows.  The U fragments and E values of the
// wave's next step are loaded while the current step computes (two register
// buffers).
// ===========================================================================
template <int KS2, int TG, bool HAS_E, bool KFULL32, bool ROT = false, bool NT = false>
__global__ __launch_bounds__(256) void decompress_mfma_bf16(
    const float* __restrict__ Zc, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ E, const uint16_t* __restrict__ U,
    uint16_t* __restrict__ Y, int64_t N, int d, int k, int64_t V) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int64_t tokb = (int64_t)blockIdx.x * (16 * TG);

  u32x4 zhi[TG][KS2], zlo[TG][KS2];
  const uint16_t* erow[TG];
  uint16_t* yrow[TG];
  bool tok_ok[TG];
#pragma unroll
  for (int tg = 0; tg < TG; ++tg) {
    int64_t t = tokb + tg * 16 + n16;
    tok_ok[tg] = t < N;
    t = t < N ? t : N - 1;
    yrow[tg] = Y + t * d + 8 * g;
    erow[tg] = HAS_E ? E + clamp_id(ids[t], V) * d + 8 * g : nullptr;
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
      split_bf16x8(v, zhi[tg][s], zlo[tg][s]);
    }
  }

  const int m4 = n16 >> 2, mr = n16 & 3;
  // A rows of tile tt: d = dbase + 32*(tt/2) + 8*(n16/4) + 4*(tt%2) + n16%4
  const uint16_t* ubase = U + (int64_t)(8 * m4 + mr) * k + 8 * g;
  const int nsteps = d >> 6;

  u32x4 ua[2][4][KS2], ev[2][TG][2];
  auto load_step = [&](int ds, u32x4(&uo)[4][KS2], u32x4(&eo)[TG][2]) {
    const int dbase = ds * 64;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      const uint16_t* up = ubase + (int64_t)(dbase + (tt >= 2 ? 32 : 0) + 4 * (tt & 1)) * k;
#pragma unroll
      for (int s = 0; s < KS2; ++s)
        uo[tt][s] = (KFULL32 || 32 * s + 8 * g < k) ? *(const u32x4*)(up + 32 * s)
                                                   : u32x4{0u, 0u, 0u, 0u};
    }
    if constexpr (HAS_E) {
#pragma unroll
      for (int tg = 0; tg < TG; ++tg) {
        eo[tg][0] = ldg<NT>(erow[tg] + dbase);
        eo[tg][1] = ldg<NT>(erow[tg] + dbase + 32);
      }
    }
  };
  auto compute_step = [&](int ds, const u32x4(&ui)[4][KS2], const u32x4(&ei)[TG][2]) {
    const int dbase = ds * 64;
#pragma unroll
    for (int tg = 0; tg < TG; ++tg) {
      f32x4 acc[4];
      if constexpr (HAS_E) {
        const u32x4 e0 = ei[tg][0], e1 = ei[tg][1];
        acc[0] = f32x4{lo_bf16(e0[0]), hi_bf16(e0[0]), lo_bf16(e0[1]), hi_bf16(e0[1])};
        acc[1] = f32x4{lo_bf16(e0[2]), hi_bf16(e0[2]), lo_bf16(e0[3]), hi_bf16(e0[3])};
        acc[2] = f32x4{lo_bf16(e1[0]), hi_bf16(e1[0]), lo_bf16(e1[1]), hi_bf16(e1[1])};
        acc[3] = f32x4{lo_bf16(e1[2]), hi_bf16(e1[2]), lo_bf16(e1[3]), hi_bf16(e1[3])};
      } else {
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int s = 0; s < KS2; ++s) {
          acc[tt] = mfma16x16x32(ui[tt][s], zhi[tg][s], acc[tt]);
          acc[tt] = mfma16x16x32(ui[tt][s], zlo[tg][s], acc[tt]);
        }
      if (tok_ok[tg]) {
        const u32x4 o0 = u32x4{pack_bf16x2(acc[0][0], acc[0][1]), pack_bf16x2(acc[0][2], acc[0][3]),
                               pack_bf16x2(acc[1][0], acc[1][1]), pack_bf16x2(acc[1][2], acc[1][3])};
        const u32x4 o1 = u32x4{pack_bf16x2(acc[2][0], acc[2][1]), pack_bf16x2(acc[2][2], acc[2][3]),
                               pack_bf16x2(acc[3][0], acc[3][1]), pack_bf16x2(acc[3][2], acc[3][3])};
        stg<NT>(yrow[tg] + dbase, o0);
        stg<NT>(yrow[tg] + dbase + 32, o1);
      }
    }
  };

  // The block visits the d steps as a rotation of [0, nsteps) starting at its
  // own offset (spreads concurrent requests over HBM channels); wave w takes
  // positions w, w+4, ... of that sequence.
  const int rot = ROT ? (int)(blockIdx.x % (unsigned)nsteps) : 0;
  auto step_at = [&](int i) { const int x = i + rot; return x < nsteps ? x : x - nsteps; };
  int i = wave;
  if (i < nsteps) load_step(step_at(i), ua[0], ev[0]);
  for (; i < nsteps; i += 8) {
    const int i1 = i + 4;
    load_step(step_at(i1 < nsteps ? i1 : i), ua[1], ev[1]);
    compute_step(step_at(i), ua[0], ev[0]);
    if (i1 >= nsteps) break;
    const int i2 = i + 8;
    load_step(step_at(i2 < nsteps ? i2 : i1), ua[0], ev[0]);
    compute_step(step_at(i1), ua[1], ev[1]);
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
  return dtype == kBF16 && d % kCompressDC == 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

bool decompress_uses_mfma(int dtype, int64_t d, int64_t k) {
  return dtype == kBF16 && d % 64 == 0 && d <= INT32_MAX && k % 8 == 0 && k >= 8 && k <= 128;
}

template <int KP, bool HAS_E, bool KFULL, int WAVES, int KS>
static hipError_t launch_compress_v(int64_t N, int d, int k, int64_t V, const void* X,
                                    const int32_t* ids, const void* E, const void* U, float* Z,
                                    hipStream_t st) {
  const int64_t blocks = (N + 16 * WAVES - 1) / (16 * WAVES);
  hipLaunchKernelGGL((compress_mfma_bf16<KP, 1, HAS_E, KFULL, false, false, WAVES, KS>),
                     dim3((unsigned)blocks), dim3(64 * WAVES), 0, st, (const uint16_t*)X, ids,
                     (const uint16_t*)E, (const uint16_t*)U, Z, N, d, k, V);
  return hipGetLastError();
}

// 8 waves (128 tokens) per block share each staged slice of U; d chunks of
// 256 when d allows, else 128.
template <int KP, bool HAS_E>
static hipError_t launch_compress_kp(int64_t N, int d, int k, int64_t V, const void* X,
                                     const int32_t* ids, const void* E, const void* U, float* Z,
                                     hipStream_t st) {
  const bool kfull = (k == 16 * KP);
  if (d % 256 == 0)
    return kfull ? launch_compress_v<KP, HAS_E, true, 8, 8>(N, d, k, V, X, ids, E, U, Z, st)
                 : launch_compress_v<KP, HAS_E, false, 8, 8>(N, d, k, V, X, ids, E, U, Z, st);
  return kfull ? launch_compress_v<KP, HAS_E, true, 8, 4>(N, d, k, V, X, ids, E, U, Z, st)
               : launch_compress_v<KP, HAS_E, false, 8, 4>(N, d, k, V, X, ids, E, U, Z, st);
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
  if (k == 32 * KS2)
    hipLaunchKernelGGL((decompress_mfma_bf16<KS2, TG, HAS_E, true, true>), dim3((unsigned)blocks),
                       dim3(256), 0, st, Zc, ids, (const uint16_t*)E, (const uint16_t*)U,
                       (uint16_t*)Y, N, d, k, V);
  else
    hipLaunchKernelGGL((decompress_mfma_bf16<KS2, TG, HAS_E, false, true>), dim3((unsigned)blocks),
                       dim3(256), 0, st, Zc, ids, (const uint16_t*)E, (const uint16_t*)U,
                       (uint16_t*)Y, N, d, k, V);
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

// Original-SSN weight re-projection W <- U (U^T W), in place.
//
// Paper: section 4.1 (the original SSN stores each output projection at full
// width and projects it back into the subspace after every optimizer step)
// and section 6.1 (re-projection happens after the optimizer step, outside the
// computational graph).  With PyTorch's [out = d, in = n] layout the rows of
// W are the constrained index, so each column w of W maps to U U^T w.
#include "ssn_device.h"
#include "ssn_launch.h"

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
  return dtype == kBF16 && d % 32 == 0 && d <= INT32_MAX && k % 8 == 0 && k >= 8 && k <= 128;
}

template <int KT>
static hipError_t launch_weights_kt(const PanelBatch& pb, int blocks, const void* U, int d, int k,
                                    hipStream_t st) {
  hipLaunchKernelGGL((project_weights_mfma_bf16<KT>), dim3(blocks), dim3(256), 0, st, pb,
                     (const uint16_t*)U, d, k);
  return hipGetLastError();
}

hipError_t launch_project_weights(int dtype, int count, int64_t d, const int64_t* n, int64_t k,
                                  void* const* W, const void* U, hipStream_t st) {
  bool aligned = (((uintptr_t)U & 15u) == 0);
  int64_t panels = 0;
  for (int b = 0; b < count; ++b) {
    aligned = aligned && (((uintptr_t)W[b] & 15u) == 0);
    panels += (n[b] + 63) / 64;
  }
  if (weights_use_mfma(dtype, d, k) && aligned && panels <= INT32_MAX) {
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

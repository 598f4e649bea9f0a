// Sparse weight averaging with the delta rule, one GPU's share (section 4.2,
// Eq. (sparta) and Eq. (delta_rule); the asynchronous sparse weight-averaging
// algorithm of section 3.3.1).  A round selects an index set P of the float32
// master weights: an index list, or a contiguous segment (the paper tiles the
// parameter vector with 20 segments and rotates through them).  The kernels
// are the memory-bound pieces of a round on one GPU:
//   snapshot    snap = theta[P]
//   average     acc = sum_r w_r c_r / sum_r w_r,  delta_r = acc - c_r
//   delta rule  theta[P] += lambda (avg - snap)
//   receive     buf[P] += lambda delta   (the same kernel without a snapshot)
// Everything streams through 16-byte accesses where the segment form and
// alignment allow, and through one 4-byte access per element otherwise.
#include "ssn_device.h"
#include "ssn_launch.h"

namespace ssn {

static unsigned stream_blocks(int64_t n, int per_thread) {
  const int64_t b = (n + 256LL * per_thread - 1) / (256LL * per_thread);
  return (unsigned)(b < 1 ? 1 : (b > 16384 ? 16384 : b));
}

// Position of the i-th selected coordinate.  List entries outside [0, n) are
// clamped into range so every access stays inside theta.
__device__ __forceinline__ int64_t sparta_pos(const int64_t* __restrict__ I, int64_t first,
                                              int64_t n, int64_t i) {
  if (!I) return first + i;
  const int64_t j = I[i];
  return j < 0 ? 0 : (j >= n ? n - 1 : j);
}

// snap[i] = theta[P_i]
__global__ __launch_bounds__(256) void sparta_gather(const float* __restrict__ theta, int64_t n,
                                                     const int64_t* __restrict__ I, int64_t first,
                                                     float* __restrict__ snap, int64_t m) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m;
       i += (int64_t)gridDim.x * blockDim.x)
    snap[i] = theta[sparta_pos(I, first, n, i)];
}

// 16-byte form of the segment snapshot (theta + first and snap 16-byte
// aligned, m % 4 == 0)
__global__ __launch_bounds__(256) void sparta_copy4(const f32x4* __restrict__ src,
                                                    f32x4* __restrict__ dst, int64_t m4) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m4;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = __builtin_nontemporal_load(src + i);
}

// theta[P_i] += lambda * (avg[i] - snap[i]); without snap, theta[P_i] += lambda * avg[i]
template <bool HAS_SNAP>
__global__ __launch_bounds__(256) void sparta_delta(float* __restrict__ theta, int64_t n,
                                                    const int64_t* __restrict__ I, int64_t first,
                                                    const float* __restrict__ avg,
                                                    const float* __restrict__ snap, float lambda,
                                                    int64_t m) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = sparta_pos(I, first, n, i);
    const float shift = HAS_SNAP ? avg[i] - snap[i] : avg[i];
    theta[j] = theta[j] + lambda * shift;
  }
}

template <bool HAS_SNAP>
__global__ __launch_bounds__(256) void sparta_delta4(f32x4* __restrict__ theta,
                                                     const f32x4* __restrict__ avg,
                                                     const f32x4* __restrict__ snap, float lambda,
                                                     int64_t m4) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m4;
       i += (int64_t)gridDim.x * blockDim.x) {
    const f32x4 a = __builtin_nontemporal_load(avg + i);
    const f32x4 s = HAS_SNAP ? __builtin_nontemporal_load(snap + i) : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 t = theta[i];
#pragma unroll
    for (int e = 0; e < 4; ++e) t[e] = t[e] + lambda * (HAS_SNAP ? a[e] - s[e] : a[e]);
    theta[i] = t;
  }
}

struct SpartaSenders {
  const float* c[kSpartaMaxSenders];
  float* delta[kSpartaMaxSenders];
  float w[kSpartaMaxSenders];
  int R;
  float inv_wsum;
};

// acc = (sum_r w_r c_r) / sum_r w_r, senders in order; delta_r = acc - c_r.
// RMAX > 0: at most RMAX senders, whose values stay in registers between the
// sum and the deltas (each chunk is read once); RMAX == 0: any count, chunks
// read again for the deltas.  V = values per thread per pass (4: 16-byte
// accesses, 1: scalar).
template <int RMAX, int V>
__global__ __launch_bounds__(256) void sparta_average(SpartaSenders s, float* __restrict__ acc,
                                                      int64_t m) {
  typedef float vec_t __attribute__((ext_vector_type(V)));
  const int64_t mv = m / V;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < mv;
       i += (int64_t)gridDim.x * blockDim.x) {
    vec_t a = (vec_t)0.f;
    if constexpr (RMAX > 0) {
      vec_t c[RMAX];
#pragma unroll
      for (int r = 0; r < RMAX; ++r)
        if (r < s.R) c[r] = __builtin_nontemporal_load((const vec_t*)s.c[r] + i);
#pragma unroll
      for (int r = 0; r < RMAX; ++r)
        if (r < s.R)
#pragma unroll
          for (int e = 0; e < V; ++e) a[e] = fmaf(s.w[r], c[r][e], a[e]);
#pragma unroll
      for (int e = 0; e < V; ++e) a[e] *= s.inv_wsum;
      __builtin_nontemporal_store(a, (vec_t*)acc + i);
#pragma unroll
      for (int r = 0; r < RMAX; ++r)
        if (r < s.R && s.delta[r]) __builtin_nontemporal_store(a - c[r], (vec_t*)s.delta[r] + i);
    } else {
      for (int r = 0; r < s.R; ++r) {
        const vec_t c = ((const vec_t*)s.c[r])[i];
#pragma unroll
        for (int e = 0; e < V; ++e) a[e] = fmaf(s.w[r], c[e], a[e]);
      }
#pragma unroll
      for (int e = 0; e < V; ++e) a[e] *= s.inv_wsum;
      ((vec_t*)acc)[i] = a;
      for (int r = 0; r < s.R; ++r)
        if (s.delta[r]) ((vec_t*)s.delta[r])[i] = a - ((const vec_t*)s.c[r])[i];
    }
  }
}

static inline bool al16f(const void* p) { return ((uintptr_t)p & 15u) == 0; }

hipError_t launch_sparta_snapshot(int64_t n, int64_t m, const int64_t* I, int64_t first, const float* theta,
                                  float* snap, hipStream_t st) {
  if (!I && m % 4 == 0 && al16f(theta + first) && al16f(snap))
    hipLaunchKernelGGL(sparta_copy4, dim3(stream_blocks(m / 4, 4)), dim3(256), 0, st,
                       (const f32x4*)(theta + first), (f32x4*)snap, m / 4);
  else
    hipLaunchKernelGGL(sparta_gather, dim3(stream_blocks(m, 4)), dim3(256), 0, st, theta, n, I,
                       first, snap, m);
  return hipGetLastError();
}

hipError_t launch_sparta_average(int R, int64_t m, const float* const* chunks, const float* weights,
                                 float* acc, float* const* deltas, hipStream_t st) {
  SpartaSenders s{};
  s.R = R;
  double wsum = 0.0;
  bool vec = (m % 4 == 0) && al16f(acc);
  for (int r = 0; r < R; ++r) {
    s.c[r] = chunks[r];
    s.delta[r] = deltas ? deltas[r] : nullptr;
    s.w[r] = weights ? weights[r] : 1.0f;
    wsum += s.w[r];
    vec = vec && al16f(s.c[r]) && (!s.delta[r] || al16f(s.delta[r]));
  }
  s.inv_wsum = (float)(1.0 / wsum);
  const int V = vec ? 4 : 1;
  const dim3 grid(stream_blocks(m / V, 4)), block(256);
#define SSN_AVG(RM, VV) hipLaunchKernelGGL((sparta_average<RM, VV>), grid, block, 0, st, s, acc, m)
  if (vec) {
    if (R <= 4) SSN_AVG(4, 4);
    else if (R <= 8) SSN_AVG(8, 4);
    else SSN_AVG(0, 4);
  } else {
    if (R <= 4) SSN_AVG(4, 1);
    else if (R <= 8) SSN_AVG(8, 1);
    else SSN_AVG(0, 1);
  }
#undef SSN_AVG
  return hipGetLastError();
}

hipError_t launch_delta_rule(int64_t n, int64_t m, const int64_t* I, int64_t first, float* theta,
                             const float* avg, const float* snap, float lambda, hipStream_t st) {
  const bool vec = !I && m % 4 == 0 && al16f(theta + first) && al16f(avg) && (!snap || al16f(snap));
  const unsigned gv = stream_blocks(m / 4, 4), gs = stream_blocks(m, 4);
  if (vec && snap)
    hipLaunchKernelGGL(sparta_delta4<true>, dim3(gv), dim3(256), 0, st, (f32x4*)(theta + first),
                       (const f32x4*)avg, (const f32x4*)snap, lambda, m / 4);
  else if (vec)
    hipLaunchKernelGGL(sparta_delta4<false>, dim3(gv), dim3(256), 0, st, (f32x4*)(theta + first),
                       (const f32x4*)avg, (const f32x4*)nullptr, lambda, m / 4);
  else if (snap)
    hipLaunchKernelGGL(sparta_delta<true>, dim3(gs), dim3(256), 0, st, theta, n, I, first, avg, snap,
                       lambda, m);
  else
    hipLaunchKernelGGL(sparta_delta<false>, dim3(gs), dim3(256), 0, st, theta, n, I, first, avg,
                       (const float*)nullptr, lambda, m);
  return hipGetLastError();
}

}  // namespace ssn

// C ABI of the codec library: argument validation (before any HIP call) and
// dispatch to the kernel launchers.  Declarations and contracts: include/ssn.h.
#include "ssn.h"

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "ssn_launch.h"

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 56;   // keeps every byte offset in int64

inline int64_t elem_size(int dtype) { return dtype == SSN_BF16 ? 2 : 4; }

inline bool aligned_to(const void* p, int64_t a) { return ((uintptr_t)p % (uintptr_t)a) == 0; }

inline bool mul_ok(int64_t a, int64_t b) { return a >= 0 && b >= 0 && (a == 0 || b <= kMaxElems / a); }

struct Span {
  uintptr_t lo, hi;
};
inline Span span(const void* p, int64_t bytes) {
  return Span{(uintptr_t)p, (uintptr_t)p + (uintptr_t)bytes};
}
inline bool overlap(Span a, Span b) {
  return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi;
}

inline ssn_status_t launch_status(hipError_t e) { return e == hipSuccess ? SSN_OK : SSN_ERR_LAUNCH; }

inline bool valid_dtype(int t) { return t == SSN_F32 || t == SSN_BF16; }

}  // namespace

extern "C" {

int ssn_abi_version(void) { return SSN_ABI_VERSION; }

const char* ssn_status_string(int status) {
  switch (status) {
    case SSN_OK: return "ok";
    case SSN_ERR_NULL: return "null pointer";
    case SSN_ERR_SHAPE: return "invalid shape";
    case SSN_ERR_DTYPE: return "invalid dtype";
    case SSN_ERR_ALIGN: return "misaligned pointer";
    case SSN_ERR_UNSUPPORTED: return "unsupported shape";
    case SSN_ERR_LAUNCH: return "kernel launch failed";
    case SSN_ERR_ALIAS: return "output overlaps an input";
    default: return "unknown status";
  }
}

const char* ssn_kernel_family(ssn_op_t op, ssn_dtype_t dtype, int64_t d, int64_t k) {
  bool mfma = false;
  switch (op) {
    case SSN_OP_COMPRESS:
    case SSN_OP_PROJECT_GRAD:
    case SSN_OP_COMPRESS_PROJECTED: mfma = ssn::compress_uses_mfma(dtype, d, k); break;
    case SSN_OP_DECOMPRESS: mfma = ssn::decompress_uses_mfma(dtype, d, k); break;
    case SSN_OP_PROJECT_WEIGHTS: mfma = ssn::weights_use_mfma(dtype, d, k); break;
    default: return "invalid";
  }
  return mfma ? "mfma" : "generic";
}

ssn_status_t ssn_compress(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                          const void* X, const int32_t* ids, const void* E, const void* U,
                          float* Z, void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || V < 1) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(V, d) || !mul_ok(d, k) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!X || !ids || !E || !U || !Z) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(X, s) || !aligned_to(E, s) || !aligned_to(U, s) || !aligned_to(ids, 4) ||
      !aligned_to(Z, 4))
    return SSN_ERR_ALIGN;
  const Span out = span(Z, N * k * 4);
  if (overlap(out, span(X, N * d * s)) || overlap(out, span(E, V * d * s)) ||
      overlap(out, span(U, d * k * s)) || overlap(out, span(ids, N * 4)))
    return SSN_ERR_ALIAS;
  return launch_status(
      ssn::launch_compress(dtype, N, d, k, V, X, ids, E, U, Z, nullptr, (hipStream_t)stream));
}

ssn_status_t ssn_compress_projected(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                                    const void* X, const int32_t* ids, const float* P,
                                    const void* U, float* Z, void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || V < 1) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(V, k) || !mul_ok(d, k) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!X || !ids || !P || !U || !Z) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(X, s) || !aligned_to(P, 4) || !aligned_to(U, s) || !aligned_to(ids, 4) ||
      !aligned_to(Z, 4))
    return SSN_ERR_ALIGN;
  const Span out = span(Z, N * k * 4);
  if (overlap(out, span(X, N * d * s)) || overlap(out, span(P, V * k * 4)) ||
      overlap(out, span(U, d * k * s)) || overlap(out, span(ids, N * 4)))
    return SSN_ERR_ALIAS;
  return launch_status(
      ssn::launch_compress(dtype, N, d, k, V, X, ids, nullptr, U, Z, P, (hipStream_t)stream));
}

ssn_status_t ssn_decompress(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                            const float* Z, const int32_t* ids, const void* E, const void* U,
                            void* Xout, void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  const bool has_e = (E != nullptr);
  if (N < 0 || d < 1 || k < 1 || k > d || (has_e && V < 1)) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(d, k) || !mul_ok(N, k) || (has_e && !mul_ok(V, d)))
    return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if ((E == nullptr) != (ids == nullptr)) return SSN_ERR_NULL;
  if (!Z || !U || !Xout) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(Z, 4) || !aligned_to(U, s) || !aligned_to(Xout, s) ||
      (has_e && (!aligned_to(E, s) || !aligned_to(ids, 4))))
    return SSN_ERR_ALIGN;
  const Span out = span(Xout, N * d * s);
  if (overlap(out, span(Z, N * k * 4)) || overlap(out, span(U, d * k * s)) ||
      (has_e && (overlap(out, span(E, V * d * s)) || overlap(out, span(ids, N * 4)))))
    return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_decompress(dtype, N, d, k, has_e ? V : 1, Z, ids, E, U, Xout,
                                              (hipStream_t)stream));
}

ssn_status_t ssn_project_grad(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, const void* G,
                              const void* U, float* GZ, void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(d, k) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!G || !U || !GZ) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(G, s) || !aligned_to(U, s) || !aligned_to(GZ, 4)) return SSN_ERR_ALIGN;
  const Span out = span(GZ, N * k * 4);
  if (overlap(out, span(G, N * d * s)) || overlap(out, span(U, d * k * s))) return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_compress(dtype, N, d, k, 1, G, nullptr, nullptr, U, GZ,
                                            nullptr, (hipStream_t)stream));
}

ssn_status_t ssn_project_table(ssn_dtype_t dtype, int64_t V, int64_t d, int64_t k, const void* E,
                               const void* U, float* P, void* stream) {
  return ssn_project_grad(dtype, V, d, k, E, U, P, stream);
}

ssn_status_t ssn_project_weights_batched(ssn_dtype_t dtype, int64_t count, int64_t d,
                                         const int64_t* n, int64_t k, void* const* W,
                                         const void* U, void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (count < 1 || count > SSN_MAX_BATCH) return SSN_ERR_SHAPE;
  if (!n || !W) return SSN_ERR_NULL;
  if (d < 1 || k < 1 || k > d || !mul_ok(d, k)) return SSN_ERR_SHAPE;
  bool any = false;
  for (int64_t b = 0; b < count; ++b) {
    if (n[b] < 0 || !mul_ok(d, n[b])) return SSN_ERR_SHAPE;
    any = any || n[b] > 0;
  }
  if (!any) return SSN_OK;
  if (k > 1024 && !ssn::weights_use_mfma(dtype, d, k)) return SSN_ERR_UNSUPPORTED;
  if (!U) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(U, s)) return SSN_ERR_ALIGN;
  const Span us = span(U, d * k * s);
  for (int64_t b = 0; b < count; ++b) {
    if (n[b] == 0) continue;
    if (!W[b]) return SSN_ERR_NULL;
    if (!aligned_to(W[b], s)) return SSN_ERR_ALIGN;
    const Span wb = span(W[b], d * n[b] * s);
    if (overlap(wb, us)) return SSN_ERR_ALIAS;
    for (int64_t c = 0; c < b; ++c)
      if (n[c] > 0 && overlap(wb, span(W[c], d * n[c] * s))) return SSN_ERR_ALIAS;
  }
  return launch_status(ssn::launch_project_weights(dtype, (int)count, d, n, k, W, U,
                                                   (hipStream_t)stream));
}

ssn_status_t ssn_project_weights(ssn_dtype_t dtype, int64_t d, int64_t n, int64_t k, void* W,
                                 const void* U, void* stream) {
  void* w[1] = {W};
  const int64_t nn[1] = {n};
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (n == 0 && d >= 1 && k >= 1 && k <= d) return SSN_OK;
  if (n > 0 && !W) return SSN_ERR_NULL;
  return ssn_project_weights_batched(dtype, 1, d, nn, k, w, U, stream);
}

}  // extern "C"

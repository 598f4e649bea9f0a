// C ABI of the codec library: argument validation (before any HIP call) and
// dispatch to the kernel launchers.  Declarations and contracts: include/ssn.h.
#include "ssn.h"

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "ssn_launch.h"
#include "ssn_checks.h"

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 56;   // keeps every byte offset in int64
// ranges of the inner dimension in the reparameterized layer's first projection
constexpr int kReparamMaxRanges = 16;

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
    case SSN_OP_COMPRESS_PROJECTED:
      mfma = ssn::compress_uses_mfma(dtype, d, k) || (dtype == SSN_F32 && ssn::f32_uses_mfma(d, k));
      break;
    case SSN_OP_DECOMPRESS:
      mfma = ssn::decompress_uses_mfma(dtype, d, k) || (dtype == SSN_F32 && ssn::f32_uses_mfma(d, k));
      break;
    case SSN_OP_PROJECT_WEIGHTS:
      mfma = ssn::weights_use_mfma(dtype, d, k) || (dtype == SSN_F32 && ssn::weights_f32_uses_mfma(d, k));
      break;
    default: return "invalid";
  }
  return mfma ? "mfma" : "generic";
}

// Coordinates in float32 (Z) or bf16 (Zb): the launchers take one of the two.
static float* z_f32(ssn_dtype_t z_dtype, void* Z) { return z_dtype == SSN_F32 ? (float*)Z : nullptr; }
static uint16_t* z_b16(ssn_dtype_t z_dtype, void* Z) {
  return z_dtype == SSN_BF16 ? (uint16_t*)Z : nullptr;
}

// A basis stored with rows of ldu >= k elements (a zero-padded copy: with
// ldu a multiple of 8 the kernels take their aligned U paths for any k); the
// launchers take the U row width as their k and the coordinate count as kz.
static bool ldu_ok(int64_t k, int64_t ldu) { return ldu >= k && ldu <= (int64_t)1 << 31; }
static int kz_of(int64_t k, int64_t ldu) { return ldu == k ? 0 : (int)k; }

ssn_status_t ssn_compress_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                             int64_t k, int64_t V, const void* X, const int32_t* ids,
                             const void* E, const void* U, int64_t ldu, void* Z, void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(z_dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || V < 1 || !ldu_ok(k, ldu)) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(V, d) || !mul_ok(d, ldu) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!X || !ids || !E || !U || !Z) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype), zs = elem_size(z_dtype);
  if (!aligned_to(X, s) || !aligned_to(E, s) || !aligned_to(U, s) || !aligned_to(ids, 4) ||
      !aligned_to(Z, zs))
    return SSN_ERR_ALIGN;
  const Span out = span(Z, N * k * zs);
  if (overlap(out, span(X, N * d * s)) || overlap(out, span(E, V * d * s)) ||
      overlap(out, span(U, d * ldu * s)) || overlap(out, span(ids, N * 4)))
    return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_compress(dtype, N, d, ldu, V, X, ids, E, U, z_f32(z_dtype, Z),
                                            nullptr, (hipStream_t)stream, z_b16(z_dtype, Z),
                                            kz_of(k, ldu)));
}

ssn_status_t ssn_compress(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                          const void* X, const int32_t* ids, const void* E, const void* U,
                          float* Z, void* stream) {
  return ssn_compress_ex(dtype, SSN_F32, N, d, k, V, X, ids, E, U, k, Z, stream);
}

ssn_status_t ssn_compress_projected_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N,
                                       int64_t d, int64_t k, int64_t V, const void* X,
                                       const int32_t* ids, const float* P, const void* U,
                                       int64_t ldu, void* Z, void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(z_dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || V < 1 || !ldu_ok(k, ldu)) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(V, k) || !mul_ok(d, ldu) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!X || !ids || !P || !U || !Z) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype), zs = elem_size(z_dtype);
  if (!aligned_to(X, s) || !aligned_to(P, 4) || !aligned_to(U, s) || !aligned_to(ids, 4) ||
      !aligned_to(Z, zs))
    return SSN_ERR_ALIGN;
  const Span out = span(Z, N * k * zs);
  if (overlap(out, span(X, N * d * s)) || overlap(out, span(P, V * k * 4)) ||
      overlap(out, span(U, d * ldu * s)) || overlap(out, span(ids, N * 4)))
    return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_compress(dtype, N, d, ldu, V, X, ids, nullptr, U,
                                            z_f32(z_dtype, Z), P, (hipStream_t)stream,
                                            z_b16(z_dtype, Z), kz_of(k, ldu)));
}

ssn_status_t ssn_compress_projected(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                                    const void* X, const int32_t* ids, const float* P,
                                    const void* U, float* Z, void* stream) {
  return ssn_compress_projected_ex(dtype, SSN_F32, N, d, k, V, X, ids, P, U, k, Z, stream);
}

ssn_status_t ssn_decompress_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                               int64_t k, int64_t V, const void* Z, const int32_t* ids,
                               const void* E, const void* U, int64_t ldu, void* Xout,
                               void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(z_dtype)) return SSN_ERR_DTYPE;
  const bool has_e = (E != nullptr);
  if (N < 0 || d < 1 || k < 1 || k > d || (has_e && V < 1) || !ldu_ok(k, ldu)) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(d, ldu) || !mul_ok(N, k) || (has_e && !mul_ok(V, d)))
    return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if ((E == nullptr) != (ids == nullptr)) return SSN_ERR_NULL;
  if (!Z || !U || !Xout) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype), zs = elem_size(z_dtype);
  if (!aligned_to(Z, zs) || !aligned_to(U, s) || !aligned_to(Xout, s) ||
      (has_e && (!aligned_to(E, s) || !aligned_to(ids, 4))))
    return SSN_ERR_ALIGN;
  const Span out = span(Xout, N * d * s);
  if (overlap(out, span(Z, N * k * zs)) || overlap(out, span(U, d * ldu * s)) ||
      (has_e && (overlap(out, span(E, V * d * s)) || overlap(out, span(ids, N * 4)))))
    return SSN_ERR_ALIAS;
  void* zm = const_cast<void*>(Z);
  return launch_status(ssn::launch_decompress(dtype, N, d, ldu, has_e ? V : 1, z_f32(z_dtype, zm),
                                              ids, E, U, Xout, false, (hipStream_t)stream,
                                              z_b16(z_dtype, zm), kz_of(k, ldu)));
}

ssn_status_t ssn_decompress(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                            const float* Z, const int32_t* ids, const void* E, const void* U,
                            void* Xout, void* stream) {
  return ssn_decompress_ex(dtype, SSN_F32, N, d, k, V, Z, ids, E, U, k, Xout, stream);
}

ssn_status_t ssn_project_grad_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                                 int64_t k, const void* G, const void* U, int64_t ldu, void* GZ,
                                 void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(z_dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || !ldu_ok(k, ldu)) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(d, ldu) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!G || !U || !GZ) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype), zs = elem_size(z_dtype);
  if (!aligned_to(G, s) || !aligned_to(U, s) || !aligned_to(GZ, zs)) return SSN_ERR_ALIGN;
  const Span out = span(GZ, N * k * zs);
  if (overlap(out, span(G, N * d * s)) || overlap(out, span(U, d * ldu * s))) return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_compress(dtype, N, d, ldu, 1, G, nullptr, nullptr, U,
                                            z_f32(z_dtype, GZ), nullptr, (hipStream_t)stream,
                                            z_b16(z_dtype, GZ), kz_of(k, ldu)));
}

ssn_status_t ssn_project_grad(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, const void* G,
                              const void* U, float* GZ, void* stream) {
  return ssn_project_grad_ex(dtype, SSN_F32, N, d, k, G, U, k, GZ, stream);
}

// The range-split projection (partial products [S][N][k] float32 in the
// workspace, S <= kRangeMax, then a range sum).  It pays where U is large
// against each compute unit's rows of G: bf16 storage, at most 16384 tokens
// and U of 512 KiB or more.  Measured on MI355X (cold G, back-to-back calls,
// both kernels): N = 4096 / 8192 / 12288 at d = 5120, U padded to 64 columns:
// 18.8 / 26.8 / 44.8 us -> 17.2 / 23.6 / 36.3 us; N = 4096 at d = 4096, k =
// 64: 16.2 -> 15.4 us; at d = 2048 (U of 192 KiB) it gained nothing at 4096
// and 8192 tokens and lost at 12288 (19.5 -> 26.0 us).
constexpr int64_t kRangeMax = 4;
static bool ranges_pay(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t ldu) {
  return dtype == SSN_BF16 && N <= 16384 && d * ldu * 2 >= (int64_t)512 << 10;
}

size_t ssn_project_grad_workspace_bytes(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k,
                                        int64_t ldu) {
  if (!valid_dtype(dtype) || N < 1 || d < 1 || k < 1 || k > d || !ldu_ok(k, ldu)) return 0;
  if (!mul_ok(N, k) || !mul_ok(d, ldu) || !ranges_pay(dtype, N, d, ldu)) return 0;
  return (size_t)(kRangeMax * N * k * 4);
}

ssn_status_t ssn_project_grad_ws(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                                 int64_t k, const void* G, const void* U, int64_t ldu, void* GZ,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(z_dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || !ldu_ok(k, ldu)) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(d, ldu) || !mul_ok(N, k)) return SSN_ERR_SHAPE;
  if (workspace_bytes > (size_t)INT64_MAX ||
      (uintptr_t)workspace + workspace_bytes < (uintptr_t)workspace)   // past the address space
    return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!G || !U || !GZ || (workspace_bytes > 0 && !workspace)) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype), zs = elem_size(z_dtype);
  if (!aligned_to(G, s) || !aligned_to(U, s) || !aligned_to(GZ, zs) ||
      (workspace && !aligned_to(workspace, 16)))
    return SSN_ERR_ALIGN;
  const Span out = span(GZ, N * k * zs);
  if (overlap(out, span(G, N * d * s)) || overlap(out, span(U, d * ldu * s))) return SSN_ERR_ALIAS;
  if (workspace_bytes > 0) {
    const Span w = span(workspace, (int64_t)workspace_bytes);
    if (overlap(w, out) || overlap(w, span(G, N * d * s)) || overlap(w, span(U, d * ldu * s)))
      return SSN_ERR_ALIAS;
  }
  int64_t smax = 1;
  if (workspace && ranges_pay(dtype, N, d, ldu)) {
    smax = (int64_t)workspace_bytes / (N * k * 4);
    smax = smax < kRangeMax ? smax : kRangeMax;
  }
  if (smax <= 1) return ssn_project_grad_ex(dtype, z_dtype, N, d, k, G, U, ldu, GZ, stream);
  return launch_status(ssn::launch_project_ranges(dtype, N, d, ldu, G, U, z_f32(z_dtype, GZ),
                                                  (float*)workspace, (int)smax, (hipStream_t)stream,
                                                  z_b16(z_dtype, GZ), kz_of(k, ldu)));
}

ssn_status_t ssn_pad_basis(ssn_dtype_t dtype, int64_t d, int64_t k, int64_t ldu, const void* U,
                           void* Up, void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (d < 1 || k < 1 || k > d || !ldu_ok(k, ldu) || !mul_ok(d, ldu)) return SSN_ERR_SHAPE;
  if (!U || !Up) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(U, s) || !aligned_to(Up, s)) return SSN_ERR_ALIGN;
  if (overlap(span(Up, d * ldu * s), span(U, d * k * s))) return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_pad_basis(dtype, d, k, ldu, U, Up, (hipStream_t)stream));
}

ssn_status_t ssn_check_ids(int64_t N, int64_t V, const int32_t* ids, int64_t* bad, void* stream) {
  if (N < 0 || V < 1 || !mul_ok(N, 4)) return SSN_ERR_SHAPE;
  if (!bad || (N > 0 && !ids)) return SSN_ERR_NULL;
  if (!aligned_to(bad, 8) || (ids && !aligned_to(ids, 4))) return SSN_ERR_ALIGN;
  if (ids && overlap(span(bad, 8), span(ids, N * 4))) return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_check_ids(N, V, ids, bad, (hipStream_t)stream));
}

ssn_status_t ssn_project_table(ssn_dtype_t dtype, int64_t V, int64_t d, int64_t k, const void* E,
                               const void* U, float* P, void* stream) {
  return ssn_project_grad(dtype, V, d, k, E, U, P, stream);
}

// ---------------------------------------------------------------------------
// Reparameterized SSN (section 4.1, Eq. (3))
// ---------------------------------------------------------------------------
static ssn_status_t reparam_shape(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d, int64_t k) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || din < 1 || d < 1 || k < 1 || k > d || k > din) return SSN_ERR_SHAPE;
  if (!mul_ok(N, din) || !mul_ok(N, d) || !mul_ok(N, k) || !mul_ok(din, k) || !mul_ok(d, k))
    return SSN_ERR_SHAPE;
  return SSN_OK;
}

// Z [N, k] = X [N, dx] . W [dx, k].  With few tokens the projection splits
// dx into ranges whose partial products go to `scratch` (row_bytes bytes per
// token, free until Z is complete) when it is large enough.
static hipError_t project_in_ranges(ssn_dtype_t dtype, int64_t N, int64_t dx, int64_t k,
                                    const void* X, const void* W, float* Z, void* scratch,
                                    int64_t row_bytes, hipStream_t st) {
  int64_t smax = aligned_to(scratch, 4) ? row_bytes / (k * 4) : 1;
  smax = smax < kReparamMaxRanges ? smax : kReparamMaxRanges;
  return ssn::launch_project_ranges(dtype, N, dx, k, X, W, Z, (float*)scratch, (int)smax, st);
}

ssn_status_t ssn_reparam_forward(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d, int64_t k,
                                 const void* H, const void* Zp, const void* U, float* T, void* Y,
                                 void* stream) {
  const ssn_status_t sh = reparam_shape(dtype, N, din, d, k);
  if (sh != SSN_OK || N == 0) return sh;
  if (!H || !Zp || !U || !T || !Y) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(H, s) || !aligned_to(Zp, s) || !aligned_to(U, s) || !aligned_to(T, 4) ||
      !aligned_to(Y, s))
    return SSN_ERR_ALIGN;
  const Span ts = span(T, N * k * 4), ys = span(Y, N * d * s);
  const Span ins[3] = {span(H, N * din * s), span(Zp, din * k * s), span(U, d * k * s)};
  for (const Span& in : ins)
    if (overlap(ts, in) || overlap(ys, in)) return SSN_ERR_ALIAS;
  if (overlap(ts, ys)) return SSN_ERR_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  // Y is written only after T is complete: it holds the partial products
  hipError_t e = project_in_ranges(dtype, N, din, k, H, Zp, T, Y, d * s, st);
  if (e != hipSuccess) return SSN_ERR_LAUNCH;
  return launch_status(ssn::launch_decompress(dtype, N, d, k, 1, T, nullptr, nullptr, U, Y, false, st));
}

size_t ssn_reparam_workspace_bytes(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t k) {
  if (!valid_dtype(dtype) || N < 0 || din < 1 || k < 1 || !mul_ok(din, k)) return 0;
  return ssn::factor_grad_workspace_bytes(dtype, N, din, k);
}

}  // extern "C"

// Arguments of ssn_reparam_backward; with check_ws false the workspace is the
// caller's business (the library's own scratch) and is not examined.
ssn_status_t ssn::reparam_backward_args(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d,
                                        int64_t k, const void* H, const void* Zp, const void* U,
                                        const void* G, const float* GT, const void* GH,
                                        const float* GZp, const void* workspace,
                                        size_t workspace_bytes, bool check_ws) {
  const ssn_status_t sh = reparam_shape(dtype, N, din, d, k);
  if (sh != SSN_OK) return sh;
  if (!GZp) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(GZp, 4)) return SSN_ERR_ALIGN;
  const size_t need = check_ws ? ssn::factor_grad_workspace_bytes(dtype, N, din, k) : 0;
  if (N > 0) {
    if (!H || !Zp || !U || !G || !GT || !GH) return SSN_ERR_NULL;
    if (!aligned_to(H, s) || !aligned_to(Zp, s) || !aligned_to(U, s) || !aligned_to(G, s) ||
        !aligned_to(GT, 4) || !aligned_to(GH, s))
      return SSN_ERR_ALIGN;
    if (workspace_bytes < need || (need > 0 && !workspace)) return SSN_ERR_SHAPE;
    if (need > 0 && !aligned_to(workspace, 4)) return SSN_ERR_ALIGN;
    const Span outs[4] = {span(GT, N * k * 4), span(GH, N * din * s), span(GZp, din * k * 4),
                          span(workspace, (int64_t)need)};
    const Span ins[4] = {span(H, N * din * s), span(Zp, din * k * s), span(U, d * k * s),
                         span(G, N * d * s)};
    for (int a = 0; a < 4; ++a) {
      for (const Span& in : ins)
        if (overlap(outs[a], in)) return SSN_ERR_ALIAS;
      for (int b = 0; b < a; ++b)
        if (overlap(outs[a], outs[b])) return SSN_ERR_ALIAS;
    }
  }
  return SSN_OK;
}

extern "C" {

ssn_status_t ssn_reparam_backward(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d, int64_t k,
                                  const void* H, const void* Zp, const void* U, const void* G,
                                  float* GT, void* GH, float* GZp, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  const ssn_status_t chk = ssn::reparam_backward_args(dtype, N, din, d, k, H, Zp, U, G, GT, GH, GZp,
                                                      workspace, workspace_bytes, true);
  if (chk != SSN_OK) return chk;
  const int64_t s = elem_size(dtype);
  hipStream_t st = (hipStream_t)stream;
  if (N == 0)   // no tokens: the factor-gradient kernel writes zeros (no memset, capture-safe)
    return launch_status(ssn::launch_factor_grad(dtype, 0, din, k, H, GT, GZp, (float*)workspace, st));
  // GH is written only after GT is complete: it holds the partial products
  hipError_t e = project_in_ranges(dtype, N, d, k, G, U, GT, GH, din * s, st);
  if (e != hipSuccess) return SSN_ERR_LAUNCH;
  if (ssn::reparam_backward_fuses(dtype, N, din, k, H, GT, Zp, GH))
    return launch_status(ssn::launch_reparam_backward_fused(N, din, k, H, GT, Zp, GH, GZp,
                                                            (float*)workspace, st));
  e = ssn::launch_decompress(dtype, N, din, k, 1, GT, nullptr, nullptr, Zp, GH, false, st);
  if (e != hipSuccess) return SSN_ERR_LAUNCH;
  return launch_status(ssn::launch_factor_grad(dtype, N, din, k, H, GT, GZp, (float*)workspace, st));
}

ssn_status_t ssn_factored_embedding(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                                    const int32_t* ids, const float* E, const void* U, void* X0,
                                    void* stream) {
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (N < 0 || d < 1 || k < 1 || k > d || V < 1) return SSN_ERR_SHAPE;
  if (!mul_ok(N, d) || !mul_ok(V, k) || !mul_ok(d, k)) return SSN_ERR_SHAPE;
  if (N == 0) return SSN_OK;
  if (!ids || !E || !U || !X0) return SSN_ERR_NULL;
  const int64_t s = elem_size(dtype);
  if (!aligned_to(ids, 4) || !aligned_to(E, 4) || !aligned_to(U, s) || !aligned_to(X0, s))
    return SSN_ERR_ALIGN;
  const Span out = span(X0, N * d * s);
  if (overlap(out, span(ids, N * 4)) || overlap(out, span(E, V * k * 4)) ||
      overlap(out, span(U, d * k * s)))
    return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_decompress(dtype, N, d, k, V, E, ids, nullptr, U, X0, true,
                                              (hipStream_t)stream));
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

size_t ssn_project_weights_workspace_bytes(int64_t d, int64_t n, int64_t k) {
  (void)d;
  (void)n;
  (void)k;
  return 0;   // U^T W stays on the compute unit that owns its columns
}

ssn_status_t ssn_project_weights(ssn_dtype_t dtype, int64_t d, int64_t n, int64_t k, void* W,
                                 const void* U, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  void* w[1] = {W};
  const int64_t nn[1] = {n};
  if (!valid_dtype(dtype)) return SSN_ERR_DTYPE;
  if (d < 1 || k < 1 || k > d || n < 0) return SSN_ERR_SHAPE;
  const size_t need = ssn_project_weights_workspace_bytes(d, n, k);
  if (workspace_bytes < need || (need > 0 && !workspace)) return SSN_ERR_SHAPE;
  if (n == 0) return SSN_OK;
  if (!W) return SSN_ERR_NULL;
  return ssn_project_weights_batched(dtype, 1, d, nn, k, w, U, stream);
}

ssn_status_t ssn_sparta_segment(int64_t n, int64_t r, int64_t segments, int64_t* first,
                                int64_t* m) {
  if (n < 0 || r < 0 || segments < 1 || segments > ((int64_t)1 << 20)) return SSN_ERR_SHAPE;
  if (!first || !m) return SSN_ERR_NULL;
  // floor(s n / S) without forming s n: n = q S + rem, so s n / S = s q + s rem / S
  const int64_t s = r % segments, q = n / segments, rem = n % segments;
  const int64_t lo = s * q + (s * rem) / segments;
  const int64_t hi = (s + 1) * q + ((s + 1) * rem) / segments;
  *first = lo;
  *m = hi - lo;
  return SSN_OK;
}

// Index set of a sparse-averaging round: the list form needs n >= 1, the
// segment form first + m <= n.
static ssn_status_t sparta_shape(int64_t n, int64_t m, const int64_t* I, int64_t first) {
  if (n < 0 || m < 0 || n > kMaxElems / 4 || m > kMaxElems / 8) return SSN_ERR_SHAPE;
  if (m == 0) return SSN_OK;
  if (I) return n >= 1 ? SSN_OK : SSN_ERR_SHAPE;
  if (first < 0 || first > n || m > n - first) return SSN_ERR_SHAPE;
  return SSN_OK;
}

ssn_status_t ssn_sparta_snapshot(int64_t n, int64_t m, const int64_t* I, int64_t first,
                                 const float* theta, float* snap, void* stream) {
  const ssn_status_t sh = sparta_shape(n, m, I, first);
  if (sh != SSN_OK || m == 0) return sh;
  if (!theta || !snap) return SSN_ERR_NULL;
  if (!aligned_to(theta, 4) || !aligned_to(snap, 4) || (I && !aligned_to(I, 8))) return SSN_ERR_ALIGN;
  const Span out = span(snap, m * 4);
  if (overlap(out, span(theta, n * 4)) || (I && overlap(out, span(I, m * 8)))) return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_sparta_snapshot(n, m, I, first, theta, snap, (hipStream_t)stream));
}

ssn_status_t ssn_sparta_average(int64_t R, int64_t m, const float* const* chunks,
                                const float* weights, float* acc, float* const* deltas,
                                void* stream) {
  if (R < 1 || R > SSN_SPARTA_MAX_SENDERS || m < 0 || m > kMaxElems / 8) return SSN_ERR_SHAPE;
  if (weights) {
    double wsum = 0.0;
    for (int64_t r = 0; r < R; ++r) {
      if (!isfinite(weights[r]) || weights[r] < 0.f) return SSN_ERR_SHAPE;
      wsum += weights[r];
    }
    if (!(wsum > 0.0) || !isfinite((float)(1.0 / wsum))) return SSN_ERR_SHAPE;
  }
  if (m == 0) return SSN_OK;
  if (!chunks || !acc) return SSN_ERR_NULL;
  if (!aligned_to(acc, 4)) return SSN_ERR_ALIGN;
  for (int64_t r = 0; r < R; ++r) {
    if (!chunks[r]) return SSN_ERR_NULL;
    if (!aligned_to(chunks[r], 4)) return SSN_ERR_ALIGN;
    if (deltas && deltas[r] && !aligned_to(deltas[r], 4)) return SSN_ERR_ALIGN;
  }
  const int64_t bytes = m * 4;
  const Span a = span(acc, bytes);
  for (int64_t r = 0; r < R; ++r) {
    const Span c = span(chunks[r], bytes);
    if (overlap(a, c)) return SSN_ERR_ALIAS;
    if (!deltas) continue;
    for (int64_t q = 0; q < R; ++q)
      if (deltas[q] && overlap(span(deltas[q], bytes), c)) return SSN_ERR_ALIAS;
    if (!deltas[r]) continue;
    const Span dr = span(deltas[r], bytes);
    if (overlap(dr, a)) return SSN_ERR_ALIAS;
    for (int64_t q = 0; q < r; ++q)
      if (deltas[q] && overlap(dr, span(deltas[q], bytes))) return SSN_ERR_ALIAS;
  }
  return launch_status(ssn::launch_sparta_average((int)R, m, chunks, weights, acc, deltas,
                                                  (hipStream_t)stream));
}

ssn_status_t ssn_delta_rule(int64_t n, int64_t m, const int64_t* I, int64_t first, float* theta,
                            const float* avg, const float* snap, float lambda, void* stream) {
  const ssn_status_t sh = sparta_shape(n, m, I, first);
  if (sh != SSN_OK) return sh;
  if (!isfinite(lambda)) return SSN_ERR_SHAPE;
  if (m == 0) return SSN_OK;
  if (!theta || !avg) return SSN_ERR_NULL;
  if (!aligned_to(theta, 4) || !aligned_to(avg, 4) || (snap && !aligned_to(snap, 4)) ||
      (I && !aligned_to(I, 8)))
    return SSN_ERR_ALIGN;
  const Span t = span(theta, n * 4);
  if (overlap(t, span(avg, m * 4)) || (snap && overlap(t, span(snap, m * 4))) ||
      (I && overlap(t, span(I, m * 8))))
    return SSN_ERR_ALIAS;
  return launch_status(ssn::launch_delta_rule(n, m, I, first, theta, avg, snap, lambda,
                                              (hipStream_t)stream));
}

}  // extern "C"

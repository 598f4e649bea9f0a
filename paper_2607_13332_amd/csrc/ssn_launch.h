// Host-side launchers implemented next to their kernels; the C ABI in
// ssn_api.hip validates arguments and then calls these.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssn {

constexpr int kF32 = 0;
constexpr int kBF16 = 1;
constexpr int kMaxBatch = 16;
constexpr int kSpartaMaxSenders = 64;

// Compute units of the current device (cached per device).
int device_cu_count();

bool compress_uses_mfma(int dtype, int64_t d, int64_t k);
bool decompress_uses_mfma(int dtype, int64_t d, int64_t k);
bool weights_use_mfma(int dtype, int64_t d, int64_t k);
// float32 storage on the matrix cores (v_mfma_f32_16x16x4_f32): d a multiple
// of 64 and U rows of 1 to 128 floats (rows whose width is not a multiple of
// 16 are staged element by element into a zero-padded tile).
bool f32_uses_mfma(int64_t d, int64_t k);
// float32 weight re-projection on the matrix cores: d a multiple of 32 and
// k <= 128 (plus, checked by the launcher, every n a multiple of 4 and 16-byte
// aligned U and W).
bool weights_f32_uses_mfma(int64_t d, int64_t k);
hipError_t launch_project_weights_f32(int count, int64_t d, const int64_t* n, int64_t k,
                                      float* const* W, const float* U, hipStream_t st);
// The reparameterized layer's factor gradient dZp = H^T GT in float32 on the
// matrix cores (the weight kernel's first pass over column strips of H):
// din a multiple of 4, k <= 128, H and GT 16-byte aligned (checked by the
// caller), any N.
bool factor_grad_f32_uses_mfma(int64_t N, int64_t din, int64_t k);
hipError_t launch_factor_grad_f32(int64_t N, int64_t din, int64_t k, const float* H, const float* GT,
                                  float* dZp, hipStream_t st);
// Ranges of d (grid.y) for `blocks` token blocks of the decompress kernels.
int decompress_grid_split(int64_t blocks, int chunks);
// float32 forms of launch_compress / launch_decompress (same arguments;
// only where f32_uses_mfma holds and X, E, U, Y are 16-byte aligned).
hipError_t launch_compress_f32(int64_t N, int64_t d, int64_t k, int64_t V, const float* X,
                               const int32_t* ids, const float* E, const float* U, float* Z,
                               const float* P, hipStream_t st, uint16_t* Zb, int kz);
hipError_t launch_decompress_f32(int64_t N, int64_t d, int64_t k, int64_t V, const float* Z,
                                 const int32_t* ids, const float* E, const float* U, float* Y,
                                 bool gather_z, hipStream_t st, const uint16_t* Zb, int kz);

// E non-NULL: Z = (X - E[ids]).U; P non-NULL: Z = X.U - P[ids]; neither: Z = X.U.
// Zb non-NULL: the coordinates are written to Zb in bf16 (rounded to nearest
// even) and Z is unused.  0 < kz < k: U rows are k wide but only their first
// kz columns are coordinates (a zero-padded basis); Z and P rows hold kz
// values.  kz <= 0: kz = k.
hipError_t launch_compress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const void* X,
                           const int32_t* ids, const void* E, const void* U, float* Z,
                           const float* P, hipStream_t st, uint16_t* Zb = nullptr, int kz = 0);
// Z = X.U (no E, no P).  With few tokens it may split d into up to smax
// ranges whose partial products go to ws [S][N][kz] (float32, S <= smax,
// written before the result) and a second kernel adds them in range order
// into Z (float32) or Zb (bf16, rounded once); ws NULL or smax <= 1: one
// launch.  kz as for launch_compress.
hipError_t launch_project_ranges(int dtype, int64_t N, int64_t d, int64_t k, const void* X,
                                 const void* U, float* Z, float* ws, int smax, hipStream_t st,
                                 uint16_t* Zb = nullptr, int kz = 0);
// E non-NULL: Y = E[ids] + Z U^T; gather_z: Y = Z[ids] U^T; else Y = Z U^T.
// Zb non-NULL: the coordinates are read from Zb in bf16 and Z is unused.
// 0 < kz < k: Z rows hold kz coordinates for the first kz of the k columns
// of U (the rest must be zero); kz <= 0 (and gather_z): kz = k.
hipError_t launch_decompress(int dtype, int64_t N, int64_t d, int64_t k, int64_t V, const float* Z,
                             const int32_t* ids, const void* E, const void* U, void* Y,
                             bool gather_z, hipStream_t st, const uint16_t* Zb = nullptr,
                             int kz = 0);
// *bad = number of ids outside [0, V) (one block, written once; N may be 0).
hipError_t launch_check_ids(int64_t N, int64_t V, const int32_t* ids, int64_t* bad, hipStream_t st);
// Up [d, ldu] = U [d, k] with zero columns k .. ldu - 1.
hipError_t launch_pad_basis(int dtype, int64_t d, int64_t k, int64_t ldu, const void* U, void* Up,
                            hipStream_t st);
// dZp[din, k] = H[N, din]^T . GT[N, k] (float32 GT and dZp); `ws` holds the
// partial sums of the token splits (factor_grad_workspace_bytes).
size_t factor_grad_workspace_bytes(int dtype, int64_t N, int64_t din, int64_t k);
hipError_t launch_factor_grad(int dtype, int64_t N, int64_t din, int64_t k, const void* H,
                              const float* GT, float* dZp, float* ws, hipStream_t st);
// Both [N, din] gradients of the reparameterized layer in one launch (plus
// the split sum): GH = GT Zp^T and dZp = H^T GT, the same bits as
// launch_decompress(GT, Zp) and launch_factor_grad; `ws` as for
// launch_factor_grad.  Only where reparam_backward_fuses() holds.
bool reparam_backward_fuses(int dtype, int64_t N, int64_t din, int64_t k, const void* H,
                            const float* GT, const void* Zp, const void* GH);
hipError_t launch_reparam_backward_fused(int64_t N, int64_t din, int64_t k, const void* H,
                                         const float* GT, const void* Zp, void* GH, float* dZp,
                                         float* ws, hipStream_t st);
// count matrices W[b] [d, n[b]] sharing U [d, k], re-projected in place.
hipError_t launch_project_weights(int dtype, int count, int64_t d, const int64_t* n, int64_t k,
                                  void* const* W, const void* U, hipStream_t st);

// Sparse averaging round (float32): snap = theta[P]; acc and per-sender
// deltas from R chunks (host arrays; weights NULL = all 1, deltas NULL or a
// NULL entry = not written); theta[P] += lambda (avg - snap), or
// += lambda avg when snap is NULL.  P = I[0..m) when I is non-NULL, else
// [first, first + m).
hipError_t launch_sparta_snapshot(int64_t n, int64_t m, const int64_t* I, int64_t first,
                                  const float* theta, float* snap, hipStream_t st);
hipError_t launch_sparta_average(int R, int64_t m, const float* const* chunks, const float* weights,
                                 float* acc, float* const* deltas, hipStream_t st);
hipError_t launch_delta_rule(int64_t n, int64_t m, const int64_t* I, int64_t first, float* theta,
                             const float* avg, const float* snap, float lambda, hipStream_t st);

}  // namespace ssn

// Exercises every C-ABI entry point's host-side validation with ordinary,
// edge and hostile arguments (sizes near INT64_MAX, counts past the limits,
// NaN weights, overlapping and misaligned pointers).  Built with
// AddressSanitizer and UndefinedBehaviorSanitizer against stub launchers:
// device pointers are fake addresses that nothing dereferences, host arrays
// are real.  Exits non-zero on the first unexpected status.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "ssn.h"

extern int g_launches;

static int g_fail = 0;
#define EXPECT(call, want)                                                              \
  do {                                                                                  \
    const int got_ = (int)(call);                                                       \
    if (got_ != (int)(want)) {                                                          \
      fprintf(stderr, "line %d: %s -> %d, expected %d\n", __LINE__, #call, got_, (int)(want)); \
      ++g_fail;                                                                         \
    }                                                                                   \
  } while (0)

static void* P(uintptr_t a) { return (void*)a; }
static const int64_t BIG = INT64_MAX;

int main() {
  void* X = P(0x100000000000);
  void* E = P(0x200000000000);
  void* U = P(0x300000000000);
  float* Z = (float*)P(0x400000000000);
  const int32_t* ids = (const int32_t*)P(0x500000000000);
  void* Y = P(0x600000000000);
  float* T = (float*)P(0x700000000000);

  EXPECT(ssn_abi_version(), SSN_ABI_VERSION);
  for (int s = -3; s < 12; ++s)
    if (!ssn_status_string(s)) ++g_fail;
  for (int op = -1; op < 7; ++op)
    for (int dt = -1; dt < 3; ++dt)
      for (int64_t d : {(int64_t)0, (int64_t)96, (int64_t)4096, BIG})
        for (int64_t k : {(int64_t)0, (int64_t)51, (int64_t)200, BIG})
          if (!ssn_kernel_family((ssn_op_t)op, (ssn_dtype_t)dt, d, k)) ++g_fail;

  // ---- compress / decompress / projections ----
  const int64_t sizes[] = {-1, 0, 1, 255, 4096, (int64_t)1 << 40, BIG - 1, BIG};
  for (int64_t N : sizes)
    for (int64_t d : sizes)
      for (int64_t k : {(int64_t)-1, (int64_t)0, (int64_t)1, (int64_t)51, (int64_t)129, BIG})
        for (int dt : {SSN_F32, SSN_BF16}) {
          // statuses vary with the shape; the point is that none misbehaves
          ssn_compress((ssn_dtype_t)dt, N, d, k, 100, X, ids, E, U, Z, nullptr);
          ssn_decompress((ssn_dtype_t)dt, N, d, k, 100, Z, ids, E, U, Y, nullptr);
          ssn_decompress((ssn_dtype_t)dt, N, d, k, 100, Z, nullptr, nullptr, U, Y, nullptr);
          ssn_project_grad((ssn_dtype_t)dt, N, d, k, X, U, Z, nullptr);
          ssn_project_table((ssn_dtype_t)dt, N, d, k, E, U, Z, nullptr);
          ssn_pad_basis((ssn_dtype_t)dt, d, k, k < BIG - 16 ? k + 13 : k, U, Y, nullptr);
          ssn_compress_projected((ssn_dtype_t)dt, N, d, k, 100, X, ids, T, U, Z, nullptr);
          ssn_factored_embedding((ssn_dtype_t)dt, N, d, k, 100, ids, T, U, Y, nullptr);
          for (int zt : {(int)SSN_F32, (int)SSN_BF16, 7}) {
            ssn_compress_ex((ssn_dtype_t)dt, (ssn_dtype_t)zt, N, d, k, 100, X, ids, E, U, k, Z, nullptr);
            ssn_compress_ex((ssn_dtype_t)dt, (ssn_dtype_t)zt, N, d, k, 100, X, ids, E, U, 64, Z, nullptr);
            ssn_decompress_ex((ssn_dtype_t)dt, (ssn_dtype_t)zt, N, d, k, 100, Z, ids, E, U, 64, Y, nullptr);
            ssn_project_grad_ex((ssn_dtype_t)dt, (ssn_dtype_t)zt, N, d, k, X, U, BIG, Z, nullptr);
            ssn_project_grad_workspace_bytes((ssn_dtype_t)dt, N, d, k, k);
            for (size_t wb : {(size_t)0, (size_t)4096, (size_t)BIG, SIZE_MAX})
              ssn_project_grad_ws((ssn_dtype_t)dt, (ssn_dtype_t)zt, N, d, k, X, U, k, Z, T, wb, nullptr);
            ssn_compress_projected_ex((ssn_dtype_t)dt, (ssn_dtype_t)zt, N, d, k, 100, X, ids, T, U, k < BIG - 8 ? k + 5 : k, Z, nullptr);
          }
        }
  EXPECT(ssn_compress(SSN_BF16, 4096, 4096, 64, 131072, X, ids, E, U, Z, nullptr), SSN_OK);
  EXPECT(ssn_compress(SSN_BF16, BIG, 4096, 64, 131072, X, ids, E, U, Z, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_compress(SSN_BF16, 4096, BIG, 64, 131072, X, ids, E, U, Z, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_compress(SSN_BF16, 4096, 4096, 64, BIG, X, ids, E, U, Z, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_compress(SSN_BF16, 0, 4096, 64, 131072, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr), SSN_OK);
  EXPECT(ssn_compress((ssn_dtype_t)9, 10, 4096, 64, 100, X, ids, E, U, Z, nullptr), SSN_ERR_DTYPE);
  EXPECT(ssn_compress(SSN_BF16, 10, 4096, 64, 100, X, ids, E, U, (float*)X, nullptr), SSN_ERR_ALIAS);
  EXPECT(ssn_compress(SSN_BF16, 10, 4096, 64, 100, (char*)X + 1, ids, E, U, Z, nullptr), SSN_ERR_ALIGN);
  EXPECT(ssn_decompress(SSN_BF16, 10, 4096, 64, 100, Z, ids, nullptr, U, Y, nullptr), SSN_ERR_NULL);
  EXPECT(ssn_decompress(SSN_BF16, 10, 4096, 64, 100, Z, nullptr, nullptr, U, Y, nullptr), SSN_OK);
  // bf16 coordinates: 2-byte alignment suffices, the span is N * k * 2 bytes
  EXPECT(ssn_compress_ex(SSN_BF16, SSN_BF16, 10, 4096, 64, 100, X, ids, E, U, 64, (char*)Z + 2, nullptr), SSN_OK);
  EXPECT(ssn_compress_ex(SSN_BF16, SSN_F32, 10, 4096, 51, 100, X, ids, E, U, 64, Z, nullptr), SSN_OK);
  EXPECT(ssn_compress_ex(SSN_BF16, SSN_F32, 10, 4096, 51, 100, X, ids, E, U, 50, Z, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_compress_ex(SSN_BF16, SSN_F32, 10, 4096, 51, 100, X, ids, E, U, BIG, Z, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_compress_ex(SSN_BF16, SSN_F32, 10, 4096, 64, 100, X, ids, E, U, 64, (char*)Z + 2, nullptr), SSN_ERR_ALIGN);
  EXPECT(ssn_compress_ex(SSN_BF16, (ssn_dtype_t)5, 10, 4096, 64, 100, X, ids, E, U, 64, Z, nullptr), SSN_ERR_DTYPE);
  EXPECT(ssn_decompress_ex(SSN_BF16, SSN_BF16, 10, 4096, 64, 100, (char*)Y - 10 * 64 * 2, ids, E, U, 64, Y, nullptr), SSN_OK);
  EXPECT(ssn_decompress_ex(SSN_BF16, SSN_BF16, 10, 4096, 64, 100, (char*)Y - 10 * 64 * 2 + 2, ids, E, U, 64, Y, nullptr), SSN_ERR_ALIAS);
  EXPECT(ssn_project_grad_ex(SSN_BF16, SSN_BF16, 10, 4096, 64, X, U, 64, (char*)X - 10 * 64 * 2, nullptr), SSN_OK);
  EXPECT(ssn_project_grad_ex(SSN_BF16, SSN_BF16, 10, 4096, 64, X, U, 64, (char*)X - 10 * 64 * 2 + 2, nullptr), SSN_ERR_ALIAS);
  // gradient projection with a workspace: the range split takes two launches
  EXPECT(ssn_project_grad_workspace_bytes(SSN_BF16, 4096, 5120, 51, 64), (size_t)4 * 4096 * 51 * 4);
  EXPECT(ssn_project_grad_workspace_bytes(SSN_F32, 4096, 5120, 51, 64), (size_t)0);
  {
    const size_t wb = ssn_project_grad_workspace_bytes(SSN_BF16, 4096, 5120, 51, 64);
    const int before = g_launches;
    EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, T, wb, nullptr), SSN_OK);
    if (g_launches != before + 2) ++g_fail;
    EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, nullptr, 0, nullptr), SSN_OK);
    if (g_launches != before + 3) ++g_fail;
  }
  EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, nullptr, 16, nullptr), SSN_ERR_NULL);
  EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, T, SIZE_MAX, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, P(UINTPTR_MAX - 15), 4096, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, (char*)T + 8, 4096, nullptr), SSN_ERR_ALIGN);
  EXPECT(ssn_project_grad_ws(SSN_BF16, SSN_F32, 4096, 5120, 51, X, U, 64, Z, (char*)Z - 16, 4096, nullptr), SSN_ERR_ALIAS);

  // ---- weight re-projection: host arrays of every legal and illegal count ----
  for (int64_t count = -1; count <= SSN_MAX_BATCH + 2; ++count) {
    const size_t m = count > 0 ? (size_t)count : 1;
    std::vector<int64_t> n(m);
    std::vector<void*> W(m);
    for (size_t b = 0; b < m; ++b) {
      n[b] = (b % 3 == 0) ? 0 : 16 * (int64_t)(b + 1);
      W[b] = P(0x800000000000 + (uintptr_t)b * 0x10000000);
    }
    const int want = (count < 1 || count > SSN_MAX_BATCH) ? SSN_ERR_SHAPE : SSN_OK;
    EXPECT(ssn_project_weights_batched(SSN_BF16, count, 4096, n.data(), 64, W.data(), U, nullptr), want);
  }
  {
    int64_t n[3] = {64, BIG, 64};
    void* W[3] = {P(0x800000000000), P(0x810000000000), P(0x820000000000)};
    EXPECT(ssn_project_weights_batched(SSN_BF16, 3, 4096, n, 64, W, U, nullptr), SSN_ERR_SHAPE);
    int64_t m[2] = {64, 64};
    void* V2[2] = {P(0x800000000000), P(0x800000000000 + 64)};   // overlapping
    EXPECT(ssn_project_weights_batched(SSN_BF16, 2, 4096, m, 64, V2, U, nullptr), SSN_ERR_ALIAS);
  }
  EXPECT(ssn_pad_basis(SSN_BF16, 5120, 51, 64, U, Y, nullptr), SSN_OK);
  EXPECT(ssn_pad_basis(SSN_BF16, 5120, 51, 50, U, Y, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_pad_basis(SSN_BF16, 5120, 51, 64, U, U, nullptr), SSN_ERR_ALIAS);
  EXPECT(ssn_pad_basis(SSN_BF16, 5120, 51, 64, nullptr, Y, nullptr), SSN_ERR_NULL);
  EXPECT(ssn_pad_basis(SSN_BF16, 5120, 51, 64, U, (char*)Y + 1, nullptr), SSN_ERR_ALIGN);
  EXPECT(ssn_project_weights_workspace_bytes(4096, 14336, 64), (size_t)0);
  EXPECT(ssn_project_weights(SSN_BF16, 4096, 14336, 64, X, U, nullptr, 0, nullptr), SSN_OK);
  EXPECT(ssn_project_weights(SSN_BF16, 4096, 14336, 64, X, U, Z, 64, nullptr), SSN_OK);
  EXPECT(ssn_project_weights(SSN_BF16, BIG, 14336, 64, X, U, nullptr, 0, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_project_weights(SSN_BF16, 4096, -1, 64, X, U, nullptr, 0, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_project_weights(SSN_BF16, 4096, 0, 64, nullptr, nullptr, nullptr, 0, nullptr), SSN_OK);
  {
    int64_t f = -1, m = -1;
    EXPECT(ssn_sparta_segment(10, 1, 4, &f, &m), SSN_OK);
    EXPECT(f, (int64_t)2);
    EXPECT(m, (int64_t)3);
    EXPECT(ssn_sparta_segment(((int64_t)1 << 56) - 1, ((int64_t)1 << 62), 1 << 20, &f, &m), SSN_OK);
    EXPECT(ssn_sparta_segment(-1, 0, 20, &f, &m), SSN_ERR_SHAPE);
    EXPECT(ssn_sparta_segment(10, -1, 20, &f, &m), SSN_ERR_SHAPE);
    EXPECT(ssn_sparta_segment(10, 0, 0, &f, &m), SSN_ERR_SHAPE);
    EXPECT(ssn_sparta_segment(10, 0, (1 << 20) + 1, &f, &m), SSN_ERR_SHAPE);
    EXPECT(ssn_sparta_segment(10, 0, 20, nullptr, &m), SSN_ERR_NULL);
  }

  // ---- reparameterized layer ----
  for (int64_t N : {(int64_t)0, (int64_t)1, (int64_t)4096, BIG})
    for (int64_t din : {(int64_t)0, (int64_t)16, (int64_t)18432, BIG}) {
      ssn_reparam_forward(SSN_BF16, N, din, 5120, 51, X, E, U, T, Y, nullptr);
      const size_t ws = ssn_reparam_workspace_bytes(SSN_BF16, N, din, 51);
      ssn_reparam_backward(SSN_BF16, N, din, 5120, 51, X, E, U, Y, T, P(0x900000000000), Z,
                           P(0xa00000000000), ws, nullptr);
    }
  EXPECT(ssn_reparam_backward(SSN_BF16, 4096, 18432, 5120, 51, X, E, U, Y, T, P(0x900000000000), Z,
                              P(0xa00000000000), 0, nullptr), SSN_ERR_SHAPE);

  // ---- delta-rule averaging ----
  const int64_t n = 1000000;
  float* theta = (float*)P(0xb00000000000);
  float* snap = (float*)P(0xc00000000000);
  const int64_t* I = (const int64_t*)P(0xd00000000000);
  EXPECT(ssn_sparta_snapshot(n, 5000, nullptr, n - 5000, theta, snap, nullptr), SSN_OK);
  EXPECT(ssn_sparta_snapshot(n, 5000, nullptr, n - 4999, theta, snap, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_sparta_snapshot(n, 5000, nullptr, BIG, theta, snap, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_sparta_snapshot(BIG, 5000, nullptr, 0, theta, snap, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_sparta_snapshot(n, BIG, I, 0, theta, snap, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_sparta_snapshot(n, 5000, I, 0, theta, snap, nullptr), SSN_OK);
  for (int64_t R = -1; R <= SSN_SPARTA_MAX_SENDERS + 2; ++R) {
    const size_t m = R > 0 ? (size_t)R : 1;
    std::vector<const float*> chunks(m);
    std::vector<float*> deltas(m);
    std::vector<float> w(m);
    for (size_t r = 0; r < m; ++r) {
      chunks[r] = (const float*)P(0xe00000000000 + (uintptr_t)r * 0x100000);
      deltas[r] = (r % 2) ? nullptr : (float*)P(0xf00000000000 + (uintptr_t)r * 0x100000);
      w[r] = (r % 4 == 1) ? 0.0f : 1.0f + (float)r;
    }
    const int want = (R < 1 || R > SSN_SPARTA_MAX_SENDERS) ? SSN_ERR_SHAPE : SSN_OK;
    EXPECT(ssn_sparta_average(R, 4096, chunks.data(), w.data(), snap, deltas.data(), nullptr), want);
    EXPECT(ssn_sparta_average(R, 4096, chunks.data(), nullptr, snap, nullptr, nullptr), want);
    if (R >= 2 && R <= SSN_SPARTA_MAX_SENDERS) {
      w[R - 1] = NAN;
      EXPECT(ssn_sparta_average(R, 4096, chunks.data(), w.data(), snap, deltas.data(), nullptr), SSN_ERR_SHAPE);
      w[R - 1] = -INFINITY;
      EXPECT(ssn_sparta_average(R, 4096, chunks.data(), w.data(), snap, deltas.data(), nullptr), SSN_ERR_SHAPE);
    }
  }
  {
    const float* c2[2] = {(const float*)P(0xe00000000000), (const float*)P(0xe00000000000 + 64)};
    EXPECT(ssn_sparta_average(2, 4096, c2, nullptr, snap, nullptr, nullptr), SSN_OK);   // inputs may overlap
    float* d2[2] = {(float*)P(0xe00000000000 + 128), nullptr};
    EXPECT(ssn_sparta_average(2, 4096, c2, nullptr, snap, d2, nullptr), SSN_ERR_ALIAS);
    const float big[2] = {3.0e38f, 3.0e38f};
    EXPECT(ssn_sparta_average(2, 4096, c2, big, snap, nullptr, nullptr), SSN_OK);
  }
  EXPECT(ssn_delta_rule(n, 5000, nullptr, 0, theta, snap, nullptr, 1.0f, nullptr), SSN_OK);
  EXPECT(ssn_delta_rule(n, 5000, I, 0, theta, snap, snap, 0.5f, nullptr), SSN_OK);
  EXPECT(ssn_delta_rule(n, 5000, nullptr, 0, theta, snap, snap, NAN, nullptr), SSN_ERR_SHAPE);
  EXPECT(ssn_delta_rule(n, BIG, nullptr, 0, theta, snap, snap, 1.0f, nullptr), SSN_ERR_SHAPE);

  if (g_launches == 0) ++g_fail;
  if (g_fail) {
    fprintf(stderr, "%d unexpected results\n", g_fail);
    return 1;
  }
  printf("abi host validation ok (%d stub launches)\n", g_launches);
  return 0;
}

// float32 column-strip launches: the weight re-projection W <- U (U^T W)
// (sections 4.1 and 6.1) and the reparameterized layer's factor gradient
// dZp = H^T (G U) (section 4.1, Eq. (3)) on the matrix cores.
#include "f32_strips.h"

namespace ssn {

SSN_STRIPS_F32_KT_EXTERN(1, false);
SSN_STRIPS_F32_KT_EXTERN(2, false);
SSN_STRIPS_F32_KT_EXTERN(3, false);
SSN_STRIPS_F32_KT_EXTERN(4, false);
SSN_STRIPS_F32_KT_EXTERN(5, false);
SSN_STRIPS_F32_KT_EXTERN(6, false);
SSN_STRIPS_F32_KT_EXTERN(7, false);
SSN_STRIPS_F32_KT_EXTERN(8, false);
SSN_STRIPS_F32_KT_EXTERN(1, true);
SSN_STRIPS_F32_KT_EXTERN(2, true);
SSN_STRIPS_F32_KT_EXTERN(3, true);
SSN_STRIPS_F32_KT_EXTERN(4, true);
SSN_STRIPS_F32_KT_EXTERN(5, true);
SSN_STRIPS_F32_KT_EXTERN(6, true);
SSN_STRIPS_F32_KT_EXTERN(7, true);
SSN_STRIPS_F32_KT_EXTERN(8, true);

template <bool FG>
static hipError_t launch_strips_f32(ColumnBatchF32& cb, const float* U, int d, int k, float* fg_out,
                                    hipStream_t st) {
  // one block per compute unit while a strip fits the LDS tiles
  const int cus = device_cu_count();
  const int tpb = (cb.tiles + cus - 1) / cus, tmax = w32_max_tpb(k);
  cb.tpb = tpb < 1 ? 1 : (tpb > tmax ? tmax : tpb);
  switch ((k + 15) / 16) {
    case 1: return launch_weights_f32_kt<1, FG>(cb, U, d, k, fg_out, st);
    case 2: return launch_weights_f32_kt<2, FG>(cb, U, d, k, fg_out, st);
    case 3: return launch_weights_f32_kt<3, FG>(cb, U, d, k, fg_out, st);
    case 4: return launch_weights_f32_kt<4, FG>(cb, U, d, k, fg_out, st);
    case 5: return launch_weights_f32_kt<5, FG>(cb, U, d, k, fg_out, st);
    case 6: return launch_weights_f32_kt<6, FG>(cb, U, d, k, fg_out, st);
    case 7: return launch_weights_f32_kt<7, FG>(cb, U, d, k, fg_out, st);
    default: return launch_weights_f32_kt<8, FG>(cb, U, d, k, fg_out, st);
  }
}

bool weights_f32_uses_mfma(int64_t d, int64_t k) {
  return d % kW32Rows == 0 && d > 0 && d <= INT32_MAX && k >= 1 && k <= 128;
}

hipError_t launch_project_weights_f32(int count, int64_t d, const int64_t* n, int64_t k,
                                      float* const* W, const float* U, hipStream_t st) {
  ColumnBatchF32 cb{};
  int nb = 0;
  int32_t acc = 0;
  for (int b = 0; b < count; ++b) {
    if (n[b] == 0) continue;
    cb.W[nb] = W[b];
    cb.n[nb] = (int32_t)n[b];
    cb.first_tile[nb] = acc;
    acc += (int32_t)((n[b] + 15) / 16);
    ++nb;
  }
  if (nb == 0) return hipSuccess;
  for (int b = nb; b <= kMaxBatch; ++b) cb.first_tile[b] = acc;
  cb.count = nb;
  cb.tiles = acc;
  return launch_strips_f32<false>(cb, U, (int)d, (int)k, nullptr, st);
}

bool factor_grad_f32_uses_mfma(int64_t N, int64_t din, int64_t k) {
  return N >= 0 && N <= INT32_MAX && din >= 1 && din % 4 == 0 && din <= INT32_MAX / 2 && k >= 1 &&
         k <= 128;
}

hipError_t launch_factor_grad_f32(int64_t N, int64_t din, int64_t k, const float* H, const float* GT,
                                  float* dZp, hipStream_t st) {
  ColumnBatchF32 cb{};
  cb.W[0] = const_cast<float*>(H);    // read only: the factor-gradient mode has no second pass
  cb.n[0] = (int32_t)din;
  const int32_t tiles = (int32_t)((din + 15) / 16);
  cb.first_tile[0] = 0;
  for (int b = 1; b <= kMaxBatch; ++b) cb.first_tile[b] = tiles;
  cb.count = 1;
  cb.tiles = tiles;
  return launch_strips_f32<true>(cb, GT, (int)N, (int)k, dZp, st);
}

}  // namespace ssn

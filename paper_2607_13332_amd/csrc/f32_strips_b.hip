// Instantiations of the float32 column-strip launcher for 5..8 k tiles
// (both modes), compiled apart so that the strip kernels build in parallel.
#include "f32_strips.h"

namespace ssn {

SSN_STRIPS_F32_KT(5, false);
SSN_STRIPS_F32_KT(5, true);
SSN_STRIPS_F32_KT(6, false);
SSN_STRIPS_F32_KT(6, true);
SSN_STRIPS_F32_KT(7, false);
SSN_STRIPS_F32_KT(7, true);
SSN_STRIPS_F32_KT(8, false);
SSN_STRIPS_F32_KT(8, true);

}  // namespace ssn

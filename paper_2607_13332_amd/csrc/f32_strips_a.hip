// Instantiations of the float32 column-strip launcher for 1..4 k tiles
// (both modes), compiled apart so that the strip kernels build in parallel.
#include "f32_strips.h"

namespace ssn {

SSN_STRIPS_F32_KT(1, false);
SSN_STRIPS_F32_KT(1, true);
SSN_STRIPS_F32_KT(2, false);
SSN_STRIPS_F32_KT(2, true);
SSN_STRIPS_F32_KT(3, false);
SSN_STRIPS_F32_KT(3, true);
SSN_STRIPS_F32_KT(4, false);
SSN_STRIPS_F32_KT(4, true);

}  // namespace ssn

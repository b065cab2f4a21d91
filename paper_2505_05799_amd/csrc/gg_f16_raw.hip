// Group-GEMM kernel instance: f16 activations, single linear.
#include "group_gemm_impl.h"

namespace mxmoe {
MXMOE_GG_LAUNCHER(gg_f16_raw, MXMOE_F16, kPhaseRaw)
}  // namespace mxmoe

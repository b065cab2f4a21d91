// Group-GEMM kernel instance: f16 activations, down phase.
#include "group_gemm_impl.h"

namespace mxmoe {
MXMOE_GG_LAUNCHER(gg_f16_p1, MXMOE_F16, 1)
}  // namespace mxmoe

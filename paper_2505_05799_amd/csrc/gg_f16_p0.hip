// Group-GEMM kernel instance: f16 activations, gate|up phase.
#include "group_gemm_impl.h"

namespace mxmoe {
MXMOE_GG_LAUNCHER(gg_f16_p0, MXMOE_F16, 0)
}  // namespace mxmoe

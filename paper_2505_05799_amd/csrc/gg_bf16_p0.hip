// Group-GEMM kernel instance: bf16 activations, gate|up phase.
#include "group_gemm_impl.h"

namespace mxmoe {
MXMOE_GG_LAUNCHER(gg_bf16_p0, MXMOE_BF16, 0)
}  // namespace mxmoe

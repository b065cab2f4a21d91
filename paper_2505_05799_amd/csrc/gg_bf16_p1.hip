// Group-GEMM kernel instance: bf16 activations, down phase.
#include "group_gemm_impl.h"

namespace mxmoe {
MXMOE_GG_LAUNCHER(gg_bf16_p1, MXMOE_BF16, 1)
}  // namespace mxmoe

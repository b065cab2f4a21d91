// Group-GEMM kernel instance: bf16 activations, single linear.
#include "group_gemm_impl.h"

namespace mxmoe {
MXMOE_GG_LAUNCHER(gg_bf16_raw, MXMOE_BF16, kPhaseRaw)
}  // namespace mxmoe

// attn_fwd_bf16_general_relu.hip -- general-path bf16 kernels (per-row visible
// ranges, runtime-coefficient bias) with the relu normalisation.
#include "bf16_kernel.h"

namespace attn {

hipError_t launch_bf16_general_relu(const AttnParams& p, int head_dim, hipStream_t stream)
{
    return launch_general_norm<kNormRelu>(p, head_dim, stream);
}

}  // namespace attn

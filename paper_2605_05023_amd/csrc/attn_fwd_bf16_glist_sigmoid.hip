// attn_fwd_bf16_glist_sigmoid.hip -- general-path bf16 kernels for the global
// sliding window with a listed global set, sigmoid normalisation.
#include "bf16_kernel.h"

namespace attn {

hipError_t launch_bf16_glist_sigmoid(const AttnParams& p, int head_dim, hipStream_t stream)
{
    return launch_general_norm<kNormSigmoid, true>(p, head_dim, stream);
}

}  // namespace attn

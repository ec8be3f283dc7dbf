// attn_fwd_bf16_glist_softmax.hip -- general-path bf16 kernels for the global
// sliding window with a listed global set, softmax normalisation.
#include "bf16_kernel.h"

namespace attn {

hipError_t launch_bf16_glist_softmax(const AttnParams& p, int head_dim, hipStream_t stream)
{
    return launch_general_norm<kNormSoftmax, true>(p, head_dim, stream);
}

}  // namespace attn

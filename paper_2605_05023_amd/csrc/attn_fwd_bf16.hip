// attn_fwd_bf16.hip -- bf16 dispatcher and the head-dim-128 instantiations of
// the closed-form-mask softmax kernels (none, causal, sliding window,
// PrefixLM, with soft-cap and one of ALiBi or the relative position bias).
// Everything else runs the general-path instantiations of the
// attn_fwd_bf16_general_*.hip units.
#include "bf16_kernel.h"

namespace attn {

int bf16_block_m() { return BM; }

namespace {

template <int D, bool LEFT>
hipError_t launch_closed_form(const AttnParams& p, hipStream_t stream)
{
    const int bias = p.slopes ? kBiasAlibi : (p.relpos ? kBiasRelPos : kBiasNone);
    return with_cap(p, [&](auto cap) {
        constexpr int C = decltype(cap)::value;
        if (bias == kBiasAlibi) return launch_variant<D, C, kBiasAlibi, kNormSoftmax, false, LEFT>(p, stream);
        if (bias == kBiasRelPos) return launch_variant<D, C, kBiasRelPos, kNormSoftmax, false, LEFT>(p, stream);
        return launch_variant<D, C, kBiasNone, kNormSoftmax, false, LEFT>(p, stream);
    });
}

}  // namespace

hipError_t launch_bf16_closed_form_d128(const AttnParams& p, hipStream_t stream)
{
    // a left-bounded band (sliding window) checks both bounds on partial tiles
    return p.band.wl >= 0 ? launch_closed_form<128, true>(p, stream)
                          : launch_closed_form<128, false>(p, stream);
}

hipError_t launch_bf16(const AttnParams& p, int head_dim, hipStream_t stream)
{
    const bool closed = p.mask_kind >= 0 && p.mask_kind <= 3;  // band masks of plan.h
    const bool both_biases = p.slopes != nullptr && p.relpos != 0;
    if (p.gtok) {  // global sliding window with a listed global set
        if (p.norm == kNormRelu) return launch_bf16_glist_relu(p, head_dim, stream);
        if (p.norm == kNormSigmoid) return launch_bf16_glist_sigmoid(p, head_dim, stream);
        return launch_bf16_glist_softmax(p, head_dim, stream);
    }
    if (p.norm == kNormRelu) return launch_bf16_general_relu(p, head_dim, stream);
    if (p.norm == kNormSigmoid) return launch_bf16_general_sigmoid(p, head_dim, stream);
    if (!closed || both_biases) return launch_bf16_general_softmax(p, head_dim, stream);
    if (head_dim == 128) return launch_bf16_closed_form_d128(p, stream);
    return launch_bf16_closed_form_d64(p, stream);
}

}  // namespace attn

// attn_fwd_bf16_d64.hip -- head-dim-64 instantiations of the closed-form-mask
// softmax kernels (see attn_fwd_bf16.hip).
#include "bf16_kernel.h"

namespace attn {

namespace {

template <bool LEFT>
hipError_t closed_form_d64(const AttnParams& p, hipStream_t stream)
{
    const int bias = p.slopes ? kBiasAlibi : (p.relpos ? kBiasRelPos : kBiasNone);
    return with_cap(p, [&](auto cap) {
        constexpr int C = decltype(cap)::value;
        if (bias == kBiasAlibi) return launch_variant<64, C, kBiasAlibi, kNormSoftmax, false, LEFT>(p, stream);
        if (bias == kBiasRelPos) return launch_variant<64, C, kBiasRelPos, kNormSoftmax, false, LEFT>(p, stream);
        return launch_variant<64, C, kBiasNone, kNormSoftmax, false, LEFT>(p, stream);
    });
}

}  // namespace

hipError_t launch_bf16_closed_form_d64(const AttnParams& p, hipStream_t stream)
{
    return p.band.wl >= 0 ? closed_form_d64<true>(p, stream) : closed_form_d64<false>(p, stream);
}

}  // namespace attn

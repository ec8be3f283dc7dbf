// launch.h -- host-side entry points of the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "kernel_params.h"

namespace attn {

// bf16 inputs, fp32 accumulation; head_dim 64 or 128.
hipError_t launch_bf16(const AttnParams& p, int head_dim, hipStream_t stream);
// (query head, query row) pairs per workgroup of the bf16 kernel
int bf16_block_m();
// instantiation groups of the bf16 kernel, one translation unit each
hipError_t launch_bf16_closed_form_d128(const AttnParams& p, hipStream_t stream);
hipError_t launch_bf16_closed_form_d64(const AttnParams& p, hipStream_t stream);
hipError_t launch_bf16_general_softmax(const AttnParams& p, int head_dim, hipStream_t stream);
hipError_t launch_bf16_general_relu(const AttnParams& p, int head_dim, hipStream_t stream);
hipError_t launch_bf16_general_sigmoid(const AttnParams& p, int head_dim, hipStream_t stream);
// general path with a listed global set (global sliding window), per normalisation
hipError_t launch_bf16_glist_softmax(const AttnParams& p, int head_dim, hipStream_t stream);
hipError_t launch_bf16_glist_relu(const AttnParams& p, int head_dim, hipStream_t stream);
hipError_t launch_bf16_glist_sigmoid(const AttnParams& p, int head_dim, hipStream_t stream);

// fp32 inputs and arithmetic; head_dim 64 or 128.
hipError_t launch_f32(const AttnParams& p, int head_dim, hipStream_t stream);
int f32_block_m();

}  // namespace attn

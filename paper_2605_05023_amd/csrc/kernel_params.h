// kernel_params.h -- argument block of the attention forward kernels.
// Filled by the host launcher from a validated attn_variant_desc.
#pragma once

#include <stdint.h>

#include "plan.h"

struct AttnParams {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    float* lse;              // may be null
    const float* slopes;     // ALiBi slope per query head, or null
    const int32_t* cu_q;     // varlen prefix sums, or null for fixed length
    const int32_t* cu_k;
    int32_t batch;           // B or number of sequences
    int32_t hq, hkv, group;  // group = hq / hkv
    int32_t seqlen_q, seqlen_k;  // fixed length
    int32_t num_q_tiles;     // ceil(max query length / block_m)
    int32_t map_mode;        // workgroup order (0 natural, 1 kv-group per XCD)
    int64_t total_q;         // varlen: rows of the [Hq, total_q] LSE
    // element strides
    int64_t sq_b, sq_h, sq_s;
    int64_t sk_b, sk_h, sk_s;
    int64_t sv_b, sv_h, sv_s;
    int64_t so_b, so_h, so_s;
    KeyBand band;            // mask as a key band
    float scale;             // multiplies q . k
    float scale_log2;        // scale * log2(e)
    float softcap;           // C, 0 = off
    float softcap_pre;       // scale / C
    float softcap_post;      // C * log2(e)
};

// kernel_params.h -- argument block of the attention forward kernels.
// Filled by the host launcher from a validated attn_variant_desc.
#pragma once

#include <stdint.h>

#include "fastdiv.h"
#include "plan.h"

// Largest listed global set of the global sliding window (staged in LDS).
constexpr int kMaxGlobalList = 2048;

// Debug build (build.py --lds-poison): every kernel first fills its LDS
// buffers with all-ones bytes (NaN in bf16 and fp32, -1 as an int), so that a
// read of LDS no load or store wrote shows in the output; a correct kernel
// gives the same bits as the release build.
#ifndef ATTN_LDS_POISON
#define ATTN_LDS_POISON 0
#endif
constexpr bool kLdsPoison = ATTN_LDS_POISON != 0;

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
    // bf16: query heads per workgroup hp (1, 2 or 4, all of one kv group;
    // wave w takes head w mod hp), log2(hp), and query rows per workgroup
    // (128 / hp; fp32: 64)
    int32_t hp, hp_shift, wg_rows;
    int32_t seqlen_q, seqlen_k;  // fixed length
    int32_t num_q_tiles;     // query tiles of wg_rows rows: ceil(max query length / 128) * hp
                             // (bf16), ceil(max query length / 64) (fp32)
    int32_t map_mode;        // workgroup order (0 natural, 1 kv-group per XCD)
    int32_t q_order;         // query tiles issued 0 last-first (causal-like), 1 first-first
    int32_t chunk;           // map_mode 1: kv-head groups per chunk within an XCD
    // bf16 variable-length batches with map_mode 1 and chunk 1: the grid holds
    // only the query spans (128 rows) of each sequence (decode_packed)
    int32_t compact;
    int32_t groups_per_xcd;  // batch * hkv / 8
    int32_t items_per_tile;  // workgroups per query tile of a kv group: group / hp
    int32_t grid;            // bf16: workgroups launched
    // bf16 listed global set: the first glob_items workgroups compute the rows
    // of G, wg_rows list entries each (glob_chunks per sequence and head set)
    int32_t glob_items, glob_chunks;
    // The divisors of the workgroup-id decode, prepared for fast_div.
    // A head set is the hp query heads of one workgroup; a kv group holds
    // group / hp of them.
    FastDiv div_bh;          // batch * hq / hp                    (map_mode 0)
    FastDiv div_hq;          // hq / hp                            (map_mode 0)
    FastDiv div_chunk_items; // chunk * group / hp * num_q_tiles   (map_mode 1)
    FastDiv div_chunk_full;  // chunk * group / hp: a full chunk's (head set, group) pairs
    FastDiv div_chunk_last;  // the same for the last chunk of an XCD
    FastDiv div_group;       // group / hp
    FastDiv div_hkv;         // hkv
    int32_t last_chunk;      // index of an XCD's last chunk
    int64_t total_q;         // varlen: rows of the [Hq, total_q] LSE
    // element strides
    int64_t sq_b, sq_h, sq_s;
    int64_t sk_b, sk_h, sk_s;
    int64_t sv_b, sv_h, sv_s;
    int64_t so_b, so_h, so_s;
    KeyBand band;            // closed-form masks as a key band
    // Masks whose visible keys come from per-row data (general path).
    int32_t mask_kind;       // attn_mask_kind_t
    int32_t num_global;      // global sliding window: size of G
    const int32_t* gtok;     // G as a sorted list of positions (device), or null for
                             // positions 0..num_global-1
    const int32_t* seg;      // segment start positions (device), or null
    int32_t num_seg;
    // elements between the segment starts (global positions) of consecutive
    // sequences; 0 = one layout for all
    int64_t seg_stride, gtok_stride;
    int32_t query_start;     // causal blockwise: first test-query position
    int32_t norm;            // attn_norm_kind_t
    int32_t relpos;          // add (i' - j) to the score
    // Scores are kept in "units": base-2 logits for softmax (unit = log2 e),
    // natural values for ReLU / Sigmoid (unit = 1).
    float unit;
    float scale;             // multiplies q . k
    float scale_u;           // scale * unit
    float softcap;           // C, 0 = off
    float softcap_pre;       // scale / C
    float softcap_pre2;      // 2 log2(e) scale / C
    float softcap_post_u;    // C * unit
    // Soft-cap as an odd polynomial in the raw dot product (kCapShort kernels
    // that fold the running max; softcap_poly.h): C' tanh(scale * dot / C) =
    // dot * sum_k cap_poly[k] dot^(2k) while dot^2 <= cap_zmax.
    float cap_poly[3];
    float cap_zmax;
};

/*
 * attn.h -- C ABI of the gfx950 fused attention forward library (libattn.so).
 *
 * The library computes the forward pass of scaled-dot-product attention,
 * O = Softmax(Score(scale * Q K^T) + Mask) V (Eq. 1 of Section 2.2 and the
 * Score / Mask / Norm decomposition of Eq. 2 and Appendix A), together with
 * the natural-log row normaliser LSE_i = log sum_j exp(score_ij). It runs as
 * one fused, tiled kernel with an online softmax on an AMD Instinct MI355X
 * (gfx950). Every argument is a plain pointer or integer; no C++ or framework
 * type crosses this boundary.
 *
 * Variants carried by attn_variant_desc (Appendix A; Appendix C names the
 * first four as the expert-library built-ins):
 *   - causal mask, sliding-window mask, ALiBi bias, tanh soft-cap
 *     (Appendix A "Softcap Attention": C * tanh(S / C)),
 *   - grouped-query heads (Section 4.1 workload tuples, e.g. 64/8/128),
 *   - variable-length packed batches (cu_seqlens prefix sums).
 * Order inside the score: scale, then soft-cap, then ALiBi bias, then mask.
 *
 * Ownership: the caller allocates and owns every buffer. The library never
 * allocates, frees or keeps a user pointer beyond the enqueued kernel. All
 * buffers must stay valid until the work on `stream` has completed.
 *
 * Errors: every entry point returns ATTN_OK (0) or a negative attn_status_t.
 * Argument validation happens on the host before any HIP call, so a rejected
 * call has no side effect. Device-side preconditions (cu_seqlens contents)
 * are documented per field and are not checked by the kernel.
 *
 * Concurrency: no global mutable state; calls on different streams may run
 * concurrently. The device used is the caller's current HIP device.
 */
#ifndef ATTN_H_
#define ATTN_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ATTN_ABI_VERSION 1

typedef enum attn_dtype {
    ATTN_BF16 = 0, /* q, k, v, out are bfloat16; accumulation in fp32 */
    ATTN_FP32 = 1  /* q, k, v, out are fp32 */
} attn_dtype_t;

/*
 * Visibility of key j from query i of a sequence with Lq queries and Lk keys.
 * The query's position on the key axis is i' = i + (Lk - Lq) (bottom-right
 * alignment; i' = i when Lq == Lk).
 *   NONE           : every key 0 <= j < Lk is visible.
 *   CAUSAL         : j <= i'.
 *   SLIDING_WINDOW : i' - j <= window_left and j - i' <= window_right, where
 *                    a negative bound is unbounded. (1023, 0) keeps keys
 *                    i'-1023 .. i'; (-1, 0) is CAUSAL; (-1, -1) is NONE.
 * A row with no visible key gets O = 0 and LSE = -inf.
 */
typedef enum attn_mask_kind {
    ATTN_MASK_NONE = 0,
    ATTN_MASK_CAUSAL = 1,
    ATTN_MASK_SLIDING_WINDOW = 2
} attn_mask_kind_t;

typedef enum attn_status {
    ATTN_OK = 0,
    ATTN_ERR_NULL_PTR = -1,    /* a required pointer is NULL                   */
    ATTN_ERR_BAD_SHAPE = -2,   /* non-positive or inconsistent sizes/strides    */
    ATTN_ERR_BAD_VARIANT = -3, /* unknown mask kind, bad window or soft-cap     */
    ATTN_ERR_ALIGNMENT = -4,   /* base not 16-byte aligned, stride not multiple
                                  of 16 bytes, or head-dim stride not 1          */
    ATTN_ERR_UNSUPPORTED = -5, /* head_dim or dtype outside the compiled set    */
    ATTN_ERR_ABI = -6,         /* struct_size does not match this library      */
    ATTN_ERR_LAUNCH = -7       /* the HIP launch reported an error             */
} attn_status_t;

/*
 * Problem description. Zero-initialise, set struct_size = sizeof(*desc), then
 * fill the fields. Strides are in elements; 0 selects the contiguous default.
 *
 * Fixed length (cu_seqlens_q == NULL):
 *   q, out [batch, num_q_heads,  seqlen_q, head_dim]
 *   k, v   [batch, num_kv_heads, seqlen_k, head_dim]
 *   lse    [batch, num_q_heads,  seqlen_q] fp32, contiguous
 * Variable length (cu_seqlens_q != NULL), sequences packed along tokens:
 *   q, out [total_q, num_q_heads,  head_dim]
 *   k, v   [total_k, num_kv_heads, head_dim]
 *   lse    [num_q_heads, total_q] fp32, contiguous
 *   Sequence s owns query rows cu_seqlens_q[s] .. cu_seqlens_q[s+1]-1 and key
 *   rows cu_seqlens_k[s] .. cu_seqlens_k[s+1]-1; sequences never attend to
 *   each other. Stride fields *_b are ignored; *_s is the token stride.
 */
typedef struct attn_variant_desc {
    uint32_t struct_size;        /* sizeof(attn_variant_desc)                      */
    int32_t dtype;               /* attn_dtype_t                                   */
    int32_t batch;               /* B, or number of sequences when varlen (>= 0)   */
    int32_t num_q_heads;         /* Hq > 0                                         */
    int32_t num_kv_heads;        /* Hkv > 0, Hq % Hkv == 0; q head h reads kv head
                                    h / (Hq / Hkv) (contiguous groups)             */
    int32_t seqlen_q, seqlen_k;  /* fixed length only (>= 0)                       */
    int32_t head_dim;            /* 64 or 128                                      */
    float scale;                 /* multiplies q . k, usually 1/sqrt(head_dim)    */
    int32_t mask_kind;           /* attn_mask_kind_t                               */
    int32_t window_left;         /* SLIDING_WINDOW only; < 0 = unbounded           */
    int32_t window_right;        /* SLIDING_WINDOW only; < 0 = unbounded           */
    const float *alibi_slopes;   /* device fp32 [num_q_heads] or NULL; adds
                                    -slope_h * |i' - j| after the soft-cap         */
    float softcap;               /* 0 = off; C > 0 maps s to C * tanh(s / C)       */
    const int32_t *cu_seqlens_q; /* device int32 [batch+1] or NULL (fixed length);
                                    must start at 0, be non-decreasing and end at
                                    total_q                                       */
    const int32_t *cu_seqlens_k; /* device int32 [batch+1]; required with
                                    cu_seqlens_q, same rules, ends at total_k      */
    int32_t max_seqlen_q;        /* varlen: >= every query length (sizes the grid) */
    int32_t max_seqlen_k;        /* varlen: >= every key length                    */
    int64_t total_q, total_k;    /* varlen: packed token counts                    */
    int64_t stride_q_b, stride_q_h, stride_q_s;
    int64_t stride_k_b, stride_k_h, stride_k_s;
    int64_t stride_v_b, stride_v_h, stride_v_s;
    int64_t stride_o_b, stride_o_h, stride_o_s;
    void *stream;                /* hipStream_t to enqueue on; NULL = default      */
} attn_variant_desc;

/*
 * Enqueue the attention forward pass on desc->stream.
 *   q, k, v : device inputs (layouts above), read only
 *   out     : device output, same dtype and layout as q; may not alias inputs
 *   lse     : device fp32 output (layout above), or NULL to skip it
 * Returns ATTN_OK once the kernel is enqueued (it runs asynchronously), or an
 * error code; on error nothing was enqueued. A zero-sized problem (batch,
 * seqlen or total of 0) enqueues nothing and returns ATTN_OK.
 */
int attn_fwd(const void *q, const void *k, const void *v, void *out, float *lse,
             const attn_variant_desc *desc);

/* Static description of an error code (never NULL). */
const char *attn_status_string(int status);

/* ATTN_ABI_VERSION of the loaded library. */
int attn_abi_version(void);

/*
 * Tile plan of one query tile (host mirror of the in-kernel planner, exposed so
 * the skipping logic can be tested without a GPU). For query rows
 * [q0, q0 + rows) of a sequence with lq queries and lk keys, key tiles of
 * `block_n` keys are classified against the mask of `desc`:
 *   out[0] = first key tile touched        out[1] = first check-free tile
 *   out[2] = one past the last check-free  out[3] = one past the last touched
 * Tiles in [out[0], out[1]) and [out[2], out[3]) need the element mask; tiles
 * in [out[1], out[2]) are fully visible for every row; tiles outside
 * [out[0], out[3]) are fully masked and skipped (loop splitting, Section 3.4).
 * When no tile is touched out[0] == out[3]. Only mask_kind, window_left and
 * window_right of desc are read.
 */
int attn_plan_tiles(const attn_variant_desc *desc, int32_t q0, int32_t rows, int32_t lq,
                    int32_t lk, int32_t block_n, int32_t out[4]);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_H_ */

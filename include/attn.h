/*
 * attn.h -- C ABI of the gfx950 fused attention forward library (libattn.so).
 *
 * The library computes the forward pass of scaled-dot-product attention,
 * O = Norm(Mask(Score(scale * Q K^T))) V (Eq. 1 of Section 2.2 and the
 * Score / Mask / Norm decomposition of Eq. 2 and Appendix A). With the
 * softmax normalisation it also returns the natural-log row normaliser
 * LSE_i = log sum_j exp(score_ij). It runs as one fused, tiled kernel (an
 * online softmax for Norm = softmax) on an AMD Instinct MI355X (gfx950).
 * Every argument is a plain pointer or integer; no C++ or framework type
 * crosses this boundary.
 *
 * Variants carried by attn_variant_desc (Appendix A; Appendix C names the
 * first four as the expert-library built-ins):
 *   - causal mask, sliding-window mask, ALiBi bias, tanh soft-cap
 *     (Appendix A "Softcap Attention": C * tanh(S / C)),
 *   - grouped-query heads (Section 4.1 workload tuples, e.g. 64/8/128),
 *   - variable-length packed batches (cu_seqlens prefix sums),
 *   - the PrefixLM, Global Sliding Window, Share Question and Causal
 *     Blockwise masks, the relative-position score term (i - j), and the
 *     ReLU and Sigmoid normalisations of Appendix A.
 * Order inside the score: scale, then soft-cap, then the ALiBi and relative
 * position biases, then the mask, then the normalisation.
 *
 * Ownership: the caller allocates and owns every buffer. The library never
 * allocates, frees or keeps a user pointer beyond the enqueued kernel. All
 * buffers must stay valid until the work on `stream` has completed.
 *
 * Errors: every entry point returns ATTN_OK (0) or a negative attn_status_t.
 * Argument validation happens on the host before any HIP call, so a rejected
 * call has no side effect. Device-side preconditions (the contents of
 * cu_seqlens, segment_starts and global_tokens) are documented per field and
 * are not checked by the kernel; ATTN_FLAG_VALIDATE checks them on the host.
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

#define ATTN_ABI_VERSION 4

/* Largest attn_variant_desc.num_segments, and num_global when global_tokens
 * lists the global positions (both are staged on chip). */
#define ATTN_MAX_SEGMENTS 2048

/*
 * attn_variant_desc.flags bits.
 * ATTN_FLAG_VALIDATE: before the launch, copy cu_seqlens_q / cu_seqlens_k,
 *   segment_starts and global_tokens to the host (waiting for desc->stream)
 *   and check the device-side preconditions documented on those fields;
 *   a violation returns ATTN_ERR_BAD_SHAPE (cu_seqlens) or
 *   ATTN_ERR_BAD_VARIANT (segments, global positions) and nothing is
 *   enqueued. A debugging aid: it costs a host round trip per call.
 * ATTN_FLAG_LOG: print one line per enqueued call to stderr naming the
 *   kernel variant and its launch plan (grid, rows and heads per workgroup,
 *   workgroup order, soft-cap form), and one line for a failed launch.
 *   Nothing is printed without it.
 */
#define ATTN_FLAG_VALIDATE 1u
#define ATTN_FLAG_LOG 2u

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
 *   PREFIX_LM      : j < prefix_len, or j <= i' (Appendix A "PrefixLM": the
 *                    prefix of length L_p is keys 0 .. L_p-1, 0-based).
 *   GLOBAL_SLIDING_WINDOW : i' - j <= window_left and j - i' <= window_right
 *                    (the paper's |i - j| <= w is window_left = window_right
 *                    = w), or i' in G, or j in G, where the global set G is
 *                    the num_global positions listed in global_tokens, or
 *                    positions 0 .. num_global-1 when global_tokens is NULL
 *                    (Appendix A "Global Sliding Window").
 *   SHARE_QUESTION : positions before segment_starts[0] are the prompt Q;
 *                    segment k (positions segment_starts[k] up to the next
 *                    start, the last one up to the end) is response A_k.
 *                    Visible iff j <= i' and either both are in Q, or i' is
 *                    in A_k and j is in Q or A_k (Appendix A "Share Question
 *                    Mask").
 *   CAUSAL_BLOCKWISE : segment k is document k (positions before
 *                    segment_starts[0] form one more document). Visible iff
 *                    j <= i' and either i' >= query_start or i' and j lie in
 *                    the same document (Appendix A "Causal Blockwise Mask").
 * A row with no visible key gets O = 0 and (softmax) LSE = -inf.
 */
typedef enum attn_mask_kind {
    ATTN_MASK_NONE = 0,
    ATTN_MASK_CAUSAL = 1,
    ATTN_MASK_SLIDING_WINDOW = 2,
    ATTN_MASK_PREFIX_LM = 3,
    ATTN_MASK_GLOBAL_SLIDING_WINDOW = 4,
    ATTN_MASK_SHARE_QUESTION = 5,
    ATTN_MASK_CAUSAL_BLOCKWISE = 6
} attn_mask_kind_t;

/*
 * Norm stage (Eq. 2 and Appendix A "Normalization Variants"), with
 * L = the key length of the row's sequence (seqlen_k, or its varlen length):
 *   SOFTMAX : P_ij = exp(s_ij) / sum_j exp(s_ij); lse is written.
 *   RELU    : P_ij = ReLU(s_ij) / L; lse is not written.
 *   SIGMOID : P_ij = Sigmoid(s_ij) / L; lse is not written.
 * Masked scores are -inf, which every normalisation sends to P = 0.
 */
typedef enum attn_norm_kind {
    ATTN_NORM_SOFTMAX = 0,
    ATTN_NORM_RELU = 1,
    ATTN_NORM_SIGMOID = 2
} attn_norm_kind_t;

typedef enum attn_status {
    ATTN_OK = 0,
    ATTN_ERR_NULL_PTR = -1,    /* a required pointer is NULL                   */
    ATTN_ERR_BAD_SHAPE = -2,   /* non-positive or inconsistent sizes/strides    */
    ATTN_ERR_BAD_VARIANT = -3, /* unknown mask or norm kind, or a bad window,
                                  soft-cap, prefix or segment count            */
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
    int32_t norm_kind;           /* attn_norm_kind_t                               */
    int32_t relative_position;   /* 1: add (i' - j) to the score after the
                                    soft-cap (Appendix A "Relative Position
                                    Embeddings"); 0: off                           */
    int32_t prefix_len;          /* PREFIX_LM: L_p >= 0                             */
    int32_t num_global;          /* GLOBAL_SLIDING_WINDOW: size of G >= 0          */
    const int32_t *segment_starts; /* SHARE_QUESTION, CAUSAL_BLOCKWISE: device
                                    int32 [num_segments], strictly increasing,
                                    >= 0; positions are per sequence (varlen)     */
    int32_t num_segments;        /* 1 .. ATTN_MAX_SEGMENTS for those kinds         */
    int32_t query_start;         /* CAUSAL_BLOCKWISE: L_q >= 0                      */
    const int32_t *global_tokens; /* GLOBAL_SLIDING_WINDOW: device int32
                                    [num_global] key positions of G, strictly
                                    increasing and >= 0 (per sequence when
                                    varlen; positions past a sequence's end are
                                    ignored), num_global <= ATTN_MAX_SEGMENTS; or
                                    NULL for G = positions 0 .. num_global-1      */
    uint32_t flags;              /* ATTN_FLAG_* bits                               */
    /* Workgroup schedule overrides for tuning and tests (0 = the library's
       choice); they change the order of the work, never the result.          */
    int32_t sched_heads_per_wg;  /* bf16: query heads of one kv group per
                                    workgroup, 1, 2 or 4, dividing Hq / Hkv       */
    int32_t sched_order;         /* 1: natural order; 2: every kv group on one
                                    XCD (needs batch * Hkv a multiple of 8)      */
    int32_t sched_chunk;         /* with sched_order 2 (or the library choosing
                                    it): kv groups walked per chunk within an XCD,
                                    1 .. batch * Hkv / 8                          */
    /* Per-sequence index-mask layouts. 0: one segment_starts (global_tokens)
       array serves every sequence. Otherwise sequence s (batch entry, or packed
       sequence when varlen) reads its own num_segments (num_global) entries at
       segment_starts + s * segment_stride (global_tokens + s * global_stride),
       each array with the rules above; stride >= the entry count. A sequence
       with fewer segments or global positions pads its array with strictly
       increasing positions at or past its end (empty segments, ignored
       global positions). */
    int64_t segment_stride;      /* SHARE_QUESTION, CAUSAL_BLOCKWISE              */
    int64_t global_stride;       /* GLOBAL_SLIDING_WINDOW with global_tokens       */
} attn_variant_desc;

/*
 * Enqueue the attention forward pass on desc->stream.
 *   q, k, v : device inputs (layouts above), read only
 *   out     : device output, same dtype and layout as q; may not alias inputs
 *   lse     : device fp32 output (layout above), or NULL to skip it; only
 *             written for the softmax normalisation
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
 * When no tile is touched out[0] == out[3]. Only mask_kind, window_left,
 * window_right and prefix_len of desc are read. The kinds whose pattern comes
 * from per-position data (GLOBAL_SLIDING_WINDOW, SHARE_QUESTION,
 * CAUSAL_BLOCKWISE) are planned inside the kernel from the rows' visible
 * ranges and return ATTN_ERR_UNSUPPORTED here.
 */
int attn_plan_tiles(const attn_variant_desc *desc, int32_t q0, int32_t rows, int32_t lq,
                    int32_t lk, int32_t block_n, int32_t out[4]);

/*
 * Keys visible to query row i (0 <= i < lq) of a sequence with lk keys under
 * the mask of `desc` (host mirror of the kernels' per-row visibility, exposed
 * so the masks can be tested without a GPU): keys j < out[0] and keys
 * out[1] <= j <= out[2] (empty when out[1] > out[2]). segment_starts is a
 * HOST copy of desc->segment_starts (read only for SHARE_QUESTION and
 * CAUSAL_BLOCKWISE); desc->segment_starts itself is not read. Reads the mask
 * fields of desc only. A GLOBAL_SLIDING_WINDOW with a listed global set
 * (global_tokens != NULL) is not of this form and returns
 * ATTN_ERR_UNSUPPORTED.
 */
int attn_row_range(const attn_variant_desc *desc, const int32_t *segment_starts, int32_t i,
                   int32_t lq, int32_t lk, int32_t out[3]);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_H_ */

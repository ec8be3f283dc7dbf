// attn_api.cpp -- C ABI of libattn.so: validation, planning and dispatch.
//
// Every check runs on the host before the first HIP call, so a rejected call
// has no side effect and the error paths are testable without a GPU. Only
// ATTN_FLAG_VALIDATE reads device memory (the cu_seqlens, segment and global
// position arrays, copied to the host) before the launch.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../../include/attn.h"
#include "kernel_params.h"
#include "launch.h"
#include "row_vis.h"
#include "softcap_poly.h"

namespace {

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

// Resolve one tensor's strides (0 = contiguous default) and check them.
// Returns ATTN_OK or an error code.
int resolve_strides(int varlen, int64_t heads, int64_t seqlen, int64_t d, int64_t elt_align,
                    int64_t in_b, int64_t in_h, int64_t in_s, int64_t* out_b, int64_t* out_h,
                    int64_t* out_s)
{
    int64_t b, h, s;
    if (varlen) {
        // [T, H, D]: token stride H*D, head stride D
        b = 0;
        h = in_h ? in_h : d;
        s = in_s ? in_s : heads * d;
    } else {
        // [B, H, S, D]
        s = in_s ? in_s : d;
        h = in_h ? in_h : seqlen * d;
        b = in_b ? in_b : heads * seqlen * d;
    }
    if (h < 0 || s < 0 || b < 0) return ATTN_ERR_BAD_SHAPE;
    if (s < d && seqlen > 1) return ATTN_ERR_BAD_SHAPE;  // rows would overlap
    if ((h % elt_align) || (s % elt_align) || (b % elt_align)) return ATTN_ERR_ALIGNMENT;
    *out_b = b;
    *out_h = h;
    *out_s = s;
    return ATTN_OK;
}

// The kernels address one (sequence, head) slice with 32-bit byte offsets.
bool slice_fits(int64_t rows, int64_t stride_s, int64_t d, int64_t elt_bytes, int64_t pad_rows)
{
    if (rows <= 0) return true;
    int64_t bytes = ((rows + pad_rows) * stride_s + d) * elt_bytes;
    return bytes < (int64_t(1) << 31);
}

// Do the D-element rows of an output with these sizes and strides stay
// disjoint? Ordered by stride, every dimension must step past the whole extent
// of the ones inside it (sufficient, and what every ordinary layout meets);
// dimensions of size one are ignored. Overlapping output rows would make the
// result depend on which workgroup writes last.
bool rows_disjoint(int64_t d, int n, const int64_t* size, const int64_t* stride)
{
    int64_t sz[3], st[3];
    int m = 0;
    for (int i = 0; i < n; ++i)
        if (size[i] > 1) {
            sz[m] = size[i];
            st[m] = stride[i];
            ++m;
        }
    for (int a = 0; a < m; ++a)  // insertion sort by stride
        for (int b = a; b > 0 && st[b] < st[b - 1]; --b) {
            int64_t t = st[b]; st[b] = st[b - 1]; st[b - 1] = t;
            t = sz[b]; sz[b] = sz[b - 1]; sz[b - 1] = t;
        }
    int64_t extent = d;  // elements covered by one row
    for (int a = 0; a < m; ++a) {
        if (st[a] < extent) return false;
        extent = st[a] * (sz[a] - 1) + extent;
    }
    return true;
}

// Host copy of a device int32 array, on `stream` (ATTN_FLAG_VALIDATE only).
bool fetch_i32(const int32_t* dev, int64_t n, hipStream_t stream, std::vector<int32_t>* out)
{
    out->assign((size_t)n, 0);
    if (n == 0) return true;
    if (hipMemcpyAsync(out->data(), dev, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost,
                       stream) != hipSuccess)
        return false;
    return hipStreamSynchronize(stream) == hipSuccess;
}

bool strictly_increasing_nonneg(const std::vector<int32_t>& a)
{
    for (size_t i = 0; i < a.size(); ++i)
        if (a[i] < 0 || (i > 0 && a[i] <= a[i - 1])) return false;
    return true;
}

// ATTN_FLAG_VALIDATE: check the device-side preconditions on the host.
int validate_device_inputs(const attn_variant_desc& d, bool varlen, bool segments, bool glist)
{
    hipStream_t stream = static_cast<hipStream_t>(d.stream);
    std::vector<int32_t> a;
    if (varlen) {
        const int32_t* cus[2] = {d.cu_seqlens_q, d.cu_seqlens_k};
        const int64_t total[2] = {d.total_q, d.total_k};
        const int64_t maxlen[2] = {d.max_seqlen_q, d.max_seqlen_k};
        for (int t = 0; t < 2; ++t) {
            if (!fetch_i32(cus[t], (int64_t)d.batch + 1, stream, &a)) return ATTN_ERR_LAUNCH;
            if (a[0] != 0 || a[(size_t)d.batch] != total[t]) return ATTN_ERR_BAD_SHAPE;
            for (int32_t s = 0; s < d.batch; ++s) {
                const int64_t len = (int64_t)a[(size_t)s + 1] - a[(size_t)s];
                if (len < 0 || len > maxlen[t]) return ATTN_ERR_BAD_SHAPE;
            }
        }
    }
    // one array, or one per sequence (a stride apart)
    auto check_arrays = [&](const int32_t* base, int64_t n, int64_t stride) {
        const int64_t copies = stride > 0 ? d.batch : 1;
        for (int64_t s = 0; s < copies; ++s) {
            if (!fetch_i32(base + s * stride, n, stream, &a)) return ATTN_ERR_LAUNCH;
            if (!strictly_increasing_nonneg(a)) return ATTN_ERR_BAD_VARIANT;
        }
        return ATTN_OK;
    };
    int rc = ATTN_OK;
    if (segments) rc = check_arrays(d.segment_starts, d.num_segments, d.segment_stride);
    if (rc == ATTN_OK && glist) rc = check_arrays(d.global_tokens, d.num_global, d.global_stride);
    return rc;
}

// ATTN_FLAG_LOG: the kernel variant and launch plan of one call, on stderr
// (the variant follows the dispatch of launch_bf16 / launch_f32).
void log_plan(const attn_variant_desc& d, const AttnParams& p)
{
    static const char* masks[] = {"none", "causal", "sliding_window", "prefix_lm",
                                  "global_sliding_window", "share_question", "causal_blockwise"};
    static const char* norms[] = {"softmax", "relu", "sigmoid"};
    const bool closed = d.mask_kind >= ATTN_MASK_NONE && d.mask_kind <= ATTN_MASK_PREFIX_LM;
    const bool both = p.slopes && p.relpos;
    const char* path = p.gtok ? "general, listed global set"
                       : (d.norm_kind != ATTN_NORM_SOFTMAX || !closed || both) ? "general"
                       : p.band.wl >= 0 ? "closed-form band with a left bound"
                                        : "closed-form band, running max checked through the row sums";
    const char* cap = d.softcap <= 0.0f                          ? "off"
                      : d.softcap <= 256.0f && p.cap_zmax >= 0.0f ? "short form, polynomial where in range"
                      : d.softcap <= 256.0f                       ? "short form"
                                                                  : "exact";
    const char* order = p.map_mode == 1 ? "kv groups per XCD" : "natural";
    std::fprintf(stderr,
                 "attn_fwd: %s D=%d B=%d Hq=%d Hkv=%d %s mask=%s norm=%s alibi=%d relpos=%d "
                 "softcap=%g (%s) | %s kernel, grid %d, %d rows x %d heads per workgroup, "
                 "order %s, chunk %d%s, global-row items %d\n",
                 d.dtype == ATTN_BF16 ? "bf16" : "fp32", d.head_dim, d.batch, d.num_q_heads,
                 d.num_kv_heads, p.cu_q ? "varlen" : "fixed-length", masks[d.mask_kind],
                 norms[d.norm_kind], p.slopes != nullptr, p.relpos, (double)d.softcap, cap,
                 d.dtype == ATTN_BF16 ? path : "fp32", p.grid, p.wg_rows, p.hp, order, p.chunk,
                 p.compact ? ", packed grid" : "", p.glob_items);
}

}  // namespace

static_assert(ATTN_MAX_SEGMENTS == kMaxGlobalList, "LDS staging of the listed global set");

extern "C" int attn_abi_version(void) { return ATTN_ABI_VERSION; }

extern "C" const char* attn_status_string(int status)
{
    switch (status) {
    case ATTN_OK: return "ok";
    case ATTN_ERR_NULL_PTR: return "a required pointer is NULL";
    case ATTN_ERR_BAD_SHAPE: return "non-positive or inconsistent sizes or strides";
    case ATTN_ERR_BAD_VARIANT: return "bad mask or norm kind, window, scale, soft-cap, prefix or segments";
    case ATTN_ERR_ALIGNMENT: return "pointer or stride not 16-byte aligned";
    case ATTN_ERR_UNSUPPORTED: return "head_dim, dtype or size outside the compiled set";
    case ATTN_ERR_ABI: return "attn_variant_desc.struct_size does not match the library";
    case ATTN_ERR_LAUNCH: return "the HIP kernel launch failed";
    default: return "unknown status";
    }
}

// The band (plan.h) of the closed-form mask kinds; for the global sliding
// window it is the window part.
static KeyBand band_of(const attn_variant_desc* d)
{
    KeyBand b = {-1, -1, 0};
    switch (d->mask_kind) {
    case ATTN_MASK_CAUSAL: b.wr = 0; break;
    case ATTN_MASK_PREFIX_LM:
        b.wr = 0;
        b.pl = d->prefix_len;
        break;
    case ATTN_MASK_SLIDING_WINDOW:
    case ATTN_MASK_GLOBAL_SLIDING_WINDOW:
        b.wl = d->window_left < 0 ? -1 : d->window_left;
        b.wr = d->window_right < 0 ? -1 : d->window_right;
        break;
    default: break;
    }
    return b;
}

static bool closed_form_mask(int kind)
{
    return kind == ATTN_MASK_NONE || kind == ATTN_MASK_CAUSAL ||
           kind == ATTN_MASK_SLIDING_WINDOW || kind == ATTN_MASK_PREFIX_LM;
}

static bool segment_mask(int kind)
{
    return kind == ATTN_MASK_SHARE_QUESTION || kind == ATTN_MASK_CAUSAL_BLOCKWISE;
}

static int check_variant(const attn_variant_desc* d)
{
    if (d->mask_kind < ATTN_MASK_NONE || d->mask_kind > ATTN_MASK_CAUSAL_BLOCKWISE)
        return ATTN_ERR_BAD_VARIANT;
    if ((d->mask_kind == ATTN_MASK_SLIDING_WINDOW ||
         d->mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW) &&
        (d->window_left < -1 || d->window_right < -1))
        return ATTN_ERR_BAD_VARIANT;
    if (d->mask_kind == ATTN_MASK_PREFIX_LM && d->prefix_len < 0) return ATTN_ERR_BAD_VARIANT;
    if (d->mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW && d->num_global < 0)
        return ATTN_ERR_BAD_VARIANT;
    if (segment_mask(d->mask_kind) &&
        (d->num_segments < 1 || d->num_segments > ATTN_MAX_SEGMENTS || d->query_start < 0))
        return ATTN_ERR_BAD_VARIANT;
    if (d->norm_kind < ATTN_NORM_SOFTMAX || d->norm_kind > ATTN_NORM_SIGMOID)
        return ATTN_ERR_BAD_VARIANT;
    if (d->relative_position != 0 && d->relative_position != 1) return ATTN_ERR_BAD_VARIANT;
    if (!std::isfinite(d->scale) || !(d->scale > 0.0f)) return ATTN_ERR_BAD_VARIANT;
    if (!std::isfinite(d->softcap) || d->softcap < 0.0f) return ATTN_ERR_BAD_VARIANT;
    // the kernels scale the dot product by 2 log2(e) scale / C: it must be finite
    if (d->softcap > 0.0f && !std::isfinite(d->scale / d->softcap * (float)(2.0 * 1.4426950408889634)))
        return ATTN_ERR_BAD_VARIANT;
    if (d->mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW && d->global_tokens &&
        d->num_global > ATTN_MAX_SEGMENTS)
        return ATTN_ERR_BAD_VARIANT;
    if (d->flags & ~(ATTN_FLAG_VALIDATE | ATTN_FLAG_LOG)) return ATTN_ERR_BAD_VARIANT;
    // per-sequence layouts: whole arrays a stride apart
    if (d->segment_stride < 0 || d->global_stride < 0) return ATTN_ERR_BAD_VARIANT;
    if (segment_mask(d->mask_kind) && d->segment_stride > 0 &&
        d->segment_stride < d->num_segments)
        return ATTN_ERR_BAD_VARIANT;
    if (d->mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW && d->global_tokens &&
        d->global_stride > 0 && d->global_stride < d->num_global)
        return ATTN_ERR_BAD_VARIANT;
    return ATTN_OK;
}

extern "C" int attn_plan_tiles(const attn_variant_desc* desc, int32_t q0, int32_t rows,
                               int32_t lq, int32_t lk, int32_t block_n, int32_t out[4])
{
    if (!desc || !out) return ATTN_ERR_NULL_PTR;
    if (desc->struct_size != sizeof(attn_variant_desc)) return ATTN_ERR_ABI;
    int rc = check_variant(desc);
    if (rc != ATTN_OK) return rc;
    if (!closed_form_mask(desc->mask_kind)) return ATTN_ERR_UNSUPPORTED;
    if (block_n <= 0 || lq < 0 || lk < 0 || rows < 0 || q0 < 0) return ATTN_ERR_BAD_SHAPE;
    TilePlan p = plan_tiles(band_of(desc), q0, rows, lq, lk, block_n);
    out[0] = p.lo;
    out[1] = p.full_lo;
    out[2] = p.full_hi;
    out[3] = p.hi;
    return ATTN_OK;
}

extern "C" int attn_row_range(const attn_variant_desc* desc, const int32_t* segment_starts,
                              int32_t i, int32_t lq, int32_t lk, int32_t out[3])
{
    if (!desc || !out) return ATTN_ERR_NULL_PTR;
    if (desc->struct_size != sizeof(attn_variant_desc)) return ATTN_ERR_ABI;
    int rc = check_variant(desc);
    if (rc != ATTN_OK) return rc;
    if (segment_mask(desc->mask_kind) && !segment_starts) return ATTN_ERR_NULL_PTR;
    // a listed global set is not a prefix plus a band
    if (desc->mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW && desc->global_tokens &&
        desc->num_global > 0)
        return ATTN_ERR_UNSUPPORTED;
    if (i < 0 || i >= lq || lk < 0) return ATTN_ERR_BAD_SHAPE;
    const int32_t* seg = segment_mask(desc->mask_kind) ? segment_starts : nullptr;
    const int32_t nseg = seg ? desc->num_segments : 0;
    RowVis r = row_visibility(desc->mask_kind, band_of(desc), desc->num_global, seg, nseg,
                              desc->query_start, i, lq, lk);
    out[0] = r.pfx;
    out[1] = r.jlo;
    out[2] = r.jhi;
    return ATTN_OK;
}

extern "C" int attn_fwd(const void* q, const void* k, const void* v, void* out, float* lse,
                        const attn_variant_desc* desc)
{
    if (!desc) return ATTN_ERR_NULL_PTR;
    if (desc->struct_size != sizeof(attn_variant_desc)) return ATTN_ERR_ABI;
    const attn_variant_desc& d = *desc;
    if (d.dtype != ATTN_BF16 && d.dtype != ATTN_FP32) return ATTN_ERR_UNSUPPORTED;
    if (d.head_dim != 64 && d.head_dim != 128) return ATTN_ERR_UNSUPPORTED;
    if (d.batch < 0 || d.num_q_heads <= 0 || d.num_kv_heads <= 0) return ATTN_ERR_BAD_SHAPE;
    if (d.num_q_heads % d.num_kv_heads != 0) return ATTN_ERR_BAD_SHAPE;
    int rc = check_variant(&d);
    if (rc != ATTN_OK) return rc;
    const int varlen = d.cu_seqlens_q != nullptr;
    if (varlen && !d.cu_seqlens_k) return ATTN_ERR_NULL_PTR;
    if (!varlen && d.cu_seqlens_k) return ATTN_ERR_BAD_SHAPE;
    int64_t max_q, max_k;
    if (varlen) {
        if (d.max_seqlen_q < 0 || d.max_seqlen_k < 0 || d.total_q < 0 || d.total_k < 0)
            return ATTN_ERR_BAD_SHAPE;
        if (d.total_q > INT32_MAX || d.total_k > INT32_MAX) return ATTN_ERR_UNSUPPORTED;
        max_q = d.max_seqlen_q;
        max_k = d.max_seqlen_k;
    } else {
        if (d.seqlen_q < 0 || d.seqlen_k < 0) return ATTN_ERR_BAD_SHAPE;
        max_q = d.seqlen_q;
        max_k = d.seqlen_k;
    }
    const int64_t elt = d.dtype == ATTN_BF16 ? 2 : 4;
    const int64_t align = 16 / elt;
    const int64_t D = d.head_dim;
    AttnParams p = {};
    rc = resolve_strides(varlen, d.num_q_heads, max_q, D, align, d.stride_q_b, d.stride_q_h,
                         d.stride_q_s, &p.sq_b, &p.sq_h, &p.sq_s);
    if (rc == ATTN_OK)
        rc = resolve_strides(varlen, d.num_kv_heads, max_k, D, align, d.stride_k_b, d.stride_k_h,
                             d.stride_k_s, &p.sk_b, &p.sk_h, &p.sk_s);
    if (rc == ATTN_OK)
        rc = resolve_strides(varlen, d.num_kv_heads, max_k, D, align, d.stride_v_b, d.stride_v_h,
                             d.stride_v_s, &p.sv_b, &p.sv_h, &p.sv_s);
    if (rc == ATTN_OK)
        rc = resolve_strides(varlen, d.num_q_heads, max_q, D, align, d.stride_o_b, d.stride_o_h,
                             d.stride_o_s, &p.so_b, &p.so_h, &p.so_s);
    if (rc != ATTN_OK) return rc;
    // 32-bit offsets inside one slice, with one tile of padding past the end.
    if (!slice_fits(max_q, p.sq_s, D, elt, 128) || !slice_fits(max_k, p.sk_s, D, elt, 128) ||
        !slice_fits(max_k, p.sv_s, D, elt, 128) || !slice_fits(max_q, p.so_s, D, elt, 128))
        return ATTN_ERR_UNSUPPORTED;

    // bf16: the query heads of one kv group share a workgroup, up to four of
    // them (one 32-row block each), so every K/V tile in LDS serves all of
    // them and the workgroup's 128 (head, row) pairs span only 32 positions,
    // which leaves fewer partially visible tiles at the mask edges.
    const int group = d.num_q_heads / d.num_kv_heads;
    int hp = d.dtype != ATTN_BF16 ? 1 : group % 4 == 0 ? 4 : group % 2 == 0 ? 2 : 1;
    if (d.sched_heads_per_wg != 0) {  // tuning override: 1, 2 or 4 dividing the group
        const int h = d.sched_heads_per_wg;
        if ((h != 1 && h != 2 && h != 4) || group % h != 0 || (d.dtype != ATTN_BF16 && h != 1))
            return ATTN_ERR_BAD_VARIANT;
        hp = h;
    }
    if (d.sched_order < 0 || d.sched_order > 2) return ATTN_ERR_BAD_VARIANT;
    if (d.sched_order == 2 && ((int64_t)d.batch * d.num_kv_heads) % 8 != 0)
        return ATTN_ERR_BAD_VARIANT;
    if (d.sched_chunk < 0 || (d.sched_chunk > 0 && d.sched_order == 1))
        return ATTN_ERR_BAD_VARIANT;
    const int block_m = d.dtype == ATTN_BF16 ? attn::bf16_block_m() / hp : attn::f32_block_m();
    // a multiple of hp: the hp query tiles of one 128-row span are issued
    // together (their K/V reads then meet in the L2)
    const int64_t q_tiles = (max_q + hp * block_m - 1) / (hp * block_m) * hp;
    const int64_t blocks = q_tiles * (d.num_q_heads / hp) * (int64_t)d.batch;
    if (blocks > INT32_MAX) return ATTN_ERR_UNSUPPORTED;
    if (blocks == 0) return ATTN_OK;  // nothing to compute

    if (!q || !k || !v || !out) return ATTN_ERR_NULL_PTR;
    if (segment_mask(d.mask_kind) && !d.segment_starts) return ATTN_ERR_NULL_PTR;
    {
        // output rows must not overlap (inputs may: a broadcast K/V is fine)
        const int64_t osize[3] = {varlen ? d.total_q : (int64_t)d.batch, d.num_q_heads,
                                  varlen ? 1 : max_q};
        const int64_t ostride[3] = {varlen ? p.so_s : p.so_b, p.so_h, p.so_s};
        if (!rows_disjoint(D, 3, osize, ostride)) return ATTN_ERR_BAD_SHAPE;
    }
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
        return ATTN_ERR_ALIGNMENT;
    if ((reinterpret_cast<uintptr_t>(lse) & 3u) != 0) return ATTN_ERR_ALIGNMENT;

    p.q = q;
    p.k = k;
    p.v = v;
    p.o = out;
    p.lse = lse;
    p.slopes = d.alibi_slopes;
    p.cu_q = d.cu_seqlens_q;
    p.cu_k = d.cu_seqlens_k;
    p.batch = d.batch;
    p.hq = d.num_q_heads;
    p.hkv = d.num_kv_heads;
    p.group = group;
    p.hp = hp;
    p.hp_shift = hp == 4 ? 2 : hp == 2 ? 1 : 0;
    p.wg_rows = block_m;
    p.seqlen_q = d.seqlen_q;
    p.seqlen_k = d.seqlen_k;
    p.num_q_tiles = (int32_t)q_tiles;
    p.total_q = varlen ? d.total_q : 0;
    p.band = band_of(&d);
    p.mask_kind = d.mask_kind;
    p.num_global = d.num_global;
    p.seg = segment_mask(d.mask_kind) ? d.segment_starts : nullptr;
    p.num_seg = segment_mask(d.mask_kind) ? d.num_segments : 0;
    p.seg_stride = segment_mask(d.mask_kind) ? d.segment_stride : 0;
    p.query_start = d.query_start;
    p.norm = d.norm_kind;
    p.relpos = d.relative_position;
    // softmax runs in base 2; the other normalisations need natural scores
    p.unit = d.norm_kind == ATTN_NORM_SOFTMAX ? 1.4426950408889634f : 1.0f;
    p.scale = d.scale;
    p.scale_u = d.scale * p.unit;
    p.softcap = d.softcap;
    p.softcap_pre = d.softcap > 0.0f ? d.scale / d.softcap : 0.0f;
    p.softcap_pre2 = p.softcap_pre * (float)(2.0 * 1.4426950408889634);
    p.softcap_post_u = d.softcap * p.unit;
    {
        // Soft-cap as dot (b0 + z (b1 + z b2)), z = dot^2 (softcap_poly.h):
        // the widest tabulated range |y| <= R, y = (scale / C) dot, whose
        // error bound C' R rel stays within kCapPolyMaxErr; the polynomial
        // holds while dot^2 <= (R / s)^2.
        p.cap_zmax = -1.0f;  // no polynomial (kernels take the exact form)
        if (d.softcap > 0.0f) {
            const double sc = (double)d.scale / d.softcap, cu = (double)p.softcap_post_u;
            int f = 0;
            while (f + 1 < kCapPolyFitCount &&
                   cu * kCapPolyFits[f].r * kCapPolyFits[f].rel > kCapPolyMaxErr)
                ++f;
            const CapPolyFit& fit = kCapPolyFits[f];
            bool normal = cu * fit.r * fit.rel <= kCapPolyMaxErr;
            double sk = sc;
            for (int c = 0; c < 3; ++c) {
                p.cap_poly[c] = (float)(cu * sk * fit.a[c]);
                normal = normal && std::fabs(p.cap_poly[c]) >= 1.1754943508222875e-38;
                sk *= sc * sc;
            }
            const double zmax = (double)fit.r * fit.r / (sc * sc);
            if (normal) p.cap_zmax = zmax < 3.0e38 ? (float)zmax : 3.0e38f;
        }
    }
    // Longest tiles first: the last query tiles under causal-like masks, the
    // first ones when global rows (which see every key) sit at the start.
    p.q_order = d.mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW && d.num_global > 0 ? 1 : 0;
    // Keep each kv-head group on one XCD when the groups divide evenly. The
    // longest-first order over all groups balances best and is kept while
    // the K/V of all groups fill at most half of the 256 MB Infinity Cache;
    // beyond that (measured: 537 MB of K/V 1.39x and 254 MB 1.03x faster
    // chunked) the groups of an XCD are walked in chunks holding at least one
    // round of its workgroup slots (32 CUs x 2), so the live K/V stays cached.
    // Not for masks where a few query tiles of each group see many times the
    // keys of the rest (the global rows of the global sliding window, the
    // rows after the question of causal blockwise): a chunk's long tiles
    // would start only with their chunk and end after everything else
    // (measured unchunked at 268 MB of K/V: 1.25x and 1.03x faster).
    // Without a mask every query tile of a group reads all of its K/V at the
    // same pace, so the groups are chunked as soon as the K/V of all groups
    // an XCD holds exceed its 4 MB L2 (ALiBi + soft-cap, 8 x 16 heads of 4096
    // keys at D = 64: L2-fabric bytes 8.6x -> 1.13x the algorithmic ones,
    // 1.04x faster).
    p.map_mode = ((int64_t)d.batch * d.num_kv_heads) % 8 == 0 ? 1 : 0;
    if (d.sched_order != 0) p.map_mode = d.sched_order == 2 ? 1 : 0;
    if (d.sched_chunk > 0 && p.map_mode != 1) return ATTN_ERR_BAD_VARIANT;
    // Size of the packed grid of a bf16 variable-length batch walked one kv
    // group at a time per XCD (see below), or -1 where it cannot apply. An
    // XCD's groups hold at most ceil(hkv / 8) kv heads of any one sequence,
    // so their query tiles (128 / hp rows) number at most
    // ceil(hkv / 8) * total_q * hp / 128 + (groups per XCD).
    int64_t packed = -1;
    if (d.dtype == ATTN_BF16 && varlen && p.map_mode == 1) {
        const int64_t groups_per_xcd = ((int64_t)d.batch * d.num_kv_heads) / 8;
        const int64_t per_seq = (d.num_kv_heads + 7) / 8;
        packed = 8 * (per_seq * d.total_q * hp / 128 + groups_per_xcd) * (group / hp);
    }
    {
        const int64_t groups_per_xcd = ((int64_t)d.batch * d.num_kv_heads) / 8;
        const int64_t kv_tokens = varlen ? d.total_k : (int64_t)d.batch * d.seqlen_k;
        const int64_t kv_bytes = kv_tokens * d.num_kv_heads * D * elt * 2;
        const int64_t per_group = (int64_t)(p.group / hp) * q_tiles;  // workgroups of a kv group
        int64_t chunk = groups_per_xcd;
        const bool few_long = d.mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW ||
                              d.mask_kind == ATTN_MASK_CAUSAL_BLOCKWISE;
        const int64_t groups = (int64_t)d.batch * d.num_kv_heads;
        const bool l2_spill = d.mask_kind == ATTN_MASK_NONE && groups > 0 &&
                              kv_bytes / groups * groups_per_xcd > (int64_t)4 << 20;
        if ((kv_bytes > (int64_t)128 << 20 || l2_spill) && !few_long)
            chunk = (64 + per_group - 1) / per_group;
        // A packed batch whose padded grid would be mostly workgroups past
        // their sequence's end (lengths far below the longest) walks its
        // groups one at a time for the packed grid, whatever its K/V size:
        // each empty workgroup still costs a dispatch and a decode (511
        // sequences of 1-64 tokens beside one of 8192: 1.05M -> 22k
        // workgroups, 1.96x faster; uniform length mixes within 2 %).
        if (packed >= 0 && !few_long && 2 * packed < blocks) chunk = 1;
        if (chunk > groups_per_xcd) chunk = groups_per_xcd;
        p.chunk = (int32_t)(chunk > 0 ? chunk : 1);
    }
    if (d.sched_chunk > 0) {  // tuning override: kv groups per chunk
        const int64_t groups_per_xcd = ((int64_t)d.batch * d.num_kv_heads) / 8;
        if (d.sched_chunk > groups_per_xcd) return ATTN_ERR_BAD_VARIANT;
        p.chunk = d.sched_chunk;
    }
    // Divisors of the workgroup-id decode (all >= 1; blocks <= INT32_MAX
    // bounds every dividend).
    const int hsets = d.num_q_heads / hp, gsets = group / hp;
    p.div_bh = make_fastdiv((uint32_t)(d.batch * hsets));
    p.div_hq = make_fastdiv((uint32_t)hsets);
    p.div_group = make_fastdiv((uint32_t)gsets);
    p.div_hkv = make_fastdiv((uint32_t)d.num_kv_heads);
    p.div_chunk_items = p.div_chunk_full = p.div_chunk_last = make_fastdiv(1);
    p.last_chunk = 0;
    if (p.map_mode == 1) {
        const int64_t groups_per_xcd = ((int64_t)d.batch * d.num_kv_heads) / 8;
        const int64_t last = (groups_per_xcd + p.chunk - 1) / p.chunk - 1;
        const int64_t last_groups = groups_per_xcd - last * p.chunk;
        p.div_chunk_items = make_fastdiv((uint32_t)((int64_t)p.chunk * gsets * q_tiles));
        p.div_chunk_full = make_fastdiv((uint32_t)(p.chunk * gsets));
        p.div_chunk_last = make_fastdiv((uint32_t)(last_groups * gsets));
        p.last_chunk = (int32_t)last;
    }
    // bf16 variable-length batch walked one kv group at a time per XCD: a
    // packed grid of only the query spans each sequence has, when smaller.
    p.grid = (int32_t)blocks;
    p.compact = 0;
    p.groups_per_xcd = 0;
    p.items_per_tile = gsets;
    if (packed >= 0 && p.chunk == 1 && packed < blocks) {
        p.compact = 1;
        p.groups_per_xcd = (int32_t)(((int64_t)d.batch * d.num_kv_heads) / 8);
        p.grid = (int32_t)packed;
    }
    const bool glist = d.mask_kind == ATTN_MASK_GLOBAL_SLIDING_WINDOW && d.global_tokens &&
                       d.num_global > 0;
    p.gtok = glist ? d.global_tokens : nullptr;
    p.gtok_stride = glist ? d.global_stride : 0;
    p.glob_items = 0;
    p.glob_chunks = 1;
    if (glist && d.dtype == ATTN_BF16) {
        p.glob_chunks = (int32_t)((d.num_global + block_m - 1) / block_m);
        const int64_t items = (int64_t)d.batch * hsets * p.glob_chunks;
        if ((int64_t)p.grid + items > INT32_MAX) return ATTN_ERR_UNSUPPORTED;
        p.glob_items = (int32_t)items;
        p.grid += p.glob_items;
    }
    if (d.flags & ATTN_FLAG_VALIDATE) {
        rc = validate_device_inputs(d, varlen, segment_mask(d.mask_kind), glist);
        if (rc != ATTN_OK) return rc;
    }
    hipStream_t stream = static_cast<hipStream_t>(d.stream);
    if (d.flags & ATTN_FLAG_LOG) log_plan(d, p);
    hipError_t err = d.dtype == ATTN_BF16 ? attn::launch_bf16(p, d.head_dim, stream)
                                          : attn::launch_f32(p, d.head_dim, stream);
    if (err != hipSuccess && (d.flags & ATTN_FLAG_LOG))
        std::fprintf(stderr, "attn_fwd: launch failed: %s\n", hipGetErrorString(err));
    return err == hipSuccess ? ATTN_OK : ATTN_ERR_LAUNCH;
}

// bf16_kernel.h -- fused attention forward for bf16 inputs on gfx950 (kernel
// template; instantiated by the attn_fwd_bf16*.hip translation units).
//
// One workgroup computes BM = 128 (query head, query row) pairs of one
// sequence: four wavefronts of 32 rows each, either 128 rows of one head or,
// when query heads share a kv head (grouped-query attention), the same 32 or
// 64 rows of the four or two heads of one kv group, which then share every
// K/V tile in LDS. It streams the key/value tiles of BN keys
// (32 or 64) that the mask leaves visible through LDS, computes the scores on the
// bf16 matrix cores with fp32 accumulation, applies the score modifications
// and, on partial tiles only, the mask in registers, keeps an online softmax
// per row, and accumulates P V on the matrix cores (Eq. 1 and 2 of Section
// 2.2; the Score / Mask / Norm stages of Appendix A; loop splitting of
// Section 3.4 and block skipping of Appendix C).
//
// Layout choices for the 64-wide wavefront and v_mfma_f32_32x32x16_bf16:
//  * Scores are computed transposed, S^T = K Q^T, so a lane owns one query
//    row (lane % 32) and 16 keys per 32-key block. The row max and row sum
//    are per-lane reductions plus one exchange with lane ^ 32.
//  * K rows are fed to the A operand in the order pi(r) (bits 2 and 3 of the
//    row index swapped). The accumulator of lane half h then holds keys
//    8h..8h+7 and 16+8h..16+8h+7 of each 32-key block in registers 0..7 and
//    8..15: exactly the B-operand layout of the P V product, so P never
//    leaves the registers.
//  * K and V tiles go from global memory straight into LDS (buffer loads with
//    an LDS destination; rows past the sequence end read as zero) in their
//    natural row-major layout. The A operand of O^T = V^T P^T is assembled by
//    two LDS transpose reads (ds_read_b64_tr_b16): in each 16-lane group,
//    output lane 4a+b element f is element b of source lane a+4f, so source
//    lanes that point at four consecutive head-dim values of four key rows
//    deliver one head-dim column across four keys to each output lane.
//  * 16-byte chunks of each LDS row are XOR-swizzled with a function of the
//    key index chosen so that both the K reads (16 rows, same chunk) and the
//    transpose reads of V (4 rows x 64 bytes) cover all 64 banks once.
//  * Software pipeline per iteration j: the QK^T products of tile j+1 are
//    issued alongside the exponentials of tile j, and the P V products of
//    tile j alongside the score mods, mask and row max of tile j+1. K tiles
//    are loaded two tiles ahead and V tiles one tile ahead, so each
//    iteration needs a single barrier.
//  * Normalisations other than softmax (ReLU, Sigmoid; Appendix A) replace the
//    exponentials by the activation and drop the running max and sum; O is
//    scaled by 1/L at the end.
//  * Masks with a closed-form band (none, causal, sliding window, PrefixLM)
//    are planned in closed form. The masks built from per-position data
//    (global sliding window, share question, causal blockwise) take the
//    general path: every lane derives its row's visible keys (a prefix plus
//    a band, row_vis.h), the workgroup reduces them to at most two ranges of
//    key tiles and a fully-visible test per tile, and the loop walks those
//    ranges, masking only the partial tiles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "kernel_params.h"
#include "launch.h"
#include "row_vis.h"
#include "score_mods.h"

namespace attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int BM = 128;      // (query head, query row) pairs per workgroup
constexpr int NT = 256;      // threads per workgroup (4 waves)
// Softmax with score mods keeps a lazily updated running max: it moves only
// when a tile's max exceeds it by more than TAU (log2 units), so P <= 2^TAU.
constexpr float TAU = 8.0f;
// Softmax without score mods and without a left bound on the visible keys
// (so that a row's first tile is the workgroup's first tile, whose max sets
// the running max) does without the tile max on the common path:
// the exponentials of a tile use the running max as it stands, and a tile
// whose per-lane partial sums of P all stay within PSUM_BOUND = 2^TAU keeps
// every P <= 2^TAU as above (a larger bound would leave the dominant P further
// from 1, where its bf16 rounding enters O unmatched by the fp32 row sum).
constexpr float PSUM_BOUND = 256.0f;

// D: head dim; BN: keys per tile; CAP: kCap* (soft-cap form); BIAS: kBias*;
// NORM: kNorm*; GEN: per-row visible ranges (general mask path); LEFT: the
// band has a left bound (otherwise every row's first visible key is 0 and
// partial tiles only check the right bound, which also masks keys past the
// sequence end).
// GLIST: the global sliding window's global set is a listed set of positions
// (general path only); its keys outside a row's band are visited after the
// planned tiles as gathered tiles.
template <int D_, int BN_, int CAP_, int BIAS_, int NORM_, bool GEN_, bool LEFT_ = true,
          bool GLIST_ = false>
struct Traits {
    static constexpr int D = D_, BN = BN_;
    static constexpr bool GLIST = GLIST_;
    static_assert(!GLIST_ || GEN_, "a listed global set takes the general path");
    static constexpr int CAP = CAP_;
    static constexpr bool SOFTCAP = CAP_ != kCapOff, MODS = SOFTCAP || BIAS_ != kBiasNone;
    static constexpr int BIAS = BIAS_, NORM = NORM_;
    static constexpr bool SOFTMAX = NORM_ == kNormSoftmax, GEN = GEN_, LEFT = LEFT_ || GEN_;
    // softmax without a left bound on the visible keys: P of a tile is made
    // with the running max as it stands and checked through the row sums
    // (check_tile); the first visited tile's max starts the running max
    static constexpr bool MAXFREE = SOFTMAX && !LEFT;
    // MAXFREE with score mods: the running max is folded into every score's
    // additive constant, so the exponential takes the score as it stands
    static constexpr bool FOLD = MAXFREE && MODS;
    // ALiBi without a left bound: key tiles are visited from the workgroup's
    // diagonal (where the row maxima lie) down to the first tile, then up to
    // the last, and check-free tiles on one side of every row take |i' - j|
    // as a per-tile constant plus the key's offset
    static constexpr bool DIAG = MAXFREE && BIAS_ == kBiasAlibi;
    // FOLD with the short soft-cap form: the pipelined steps take the soft-cap
    // of a tile from an odd polynomial in the dot product while every |y| of
    // the tile (y = scale * dot / C) stays within its range, and recompute the
    // tile with the short form otherwise (fold_score)
    static constexpr bool POLY = FOLD && CAP_ == kCapShort;
    // softmax with soft-cap or ALiBi, or on the general (index-mask) path: O
    // is normalised by the sum of P as rounded to bf16 (ALiBi makes rows
    // local, index masks leave some rows few keys; there the rounding of a
    // row's largest P would show in O). The relative position term alone
    // makes a row's first visible key its largest, and that key's tile sets
    // the running max exactly.
    static constexpr bool PSUM_BF16 = SOFTMAX && (SOFTCAP || BIAS_ == kBiasAlibi || GEN);
    static constexpr int NB = BN / 32;                   // 32-key blocks per tile
    static constexpr int ROWB = D * 2;                   // bytes per K/V row in LDS
    static constexpr int TILE = BN * ROWB;               // bytes per K or V tile
    static constexpr int LOADS = TILE / (NT * 16);       // 16-byte loads per thread per tile
    static constexpr int ROWS_PER_LOAD = NT * 16 / ROWB; // tile rows covered by one load round
    static constexpr int KSTEPS = D / 16;                // MFMA k-steps over the head dim
    static constexpr int DBLK = D / 32;                  // 32-row blocks of O^T
    static_assert(BN == 32 || BN == 64, "key tile");
    static_assert(LOADS >= 1 && LOADS * NT * 16 == TILE, "tile split");
    static_assert(ROWS_PER_LOAD % 16 == 0, "swizzle period");
};

// pi: swap bits 2 and 3 of a row index within a 32-row block.
__device__ __forceinline__ int pi32(int r)
{
    return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// XOR applied to the 16-byte chunk index of key row `key` in LDS.
template <int D>
__device__ __forceinline__ int chunk_swizzle(int key)
{
    if constexpr (D == 128)
        return ((key & 3) << 2) | ((key >> 2) & 3);
    else
        return (((key >> 1) & 1) << 2) | ((key >> 2) & 3);
}

// s_waitcnt immediate that waits until at most n vector memory operations are
// outstanding and leaves the other counters unconstrained (gfx9 encoding:
// vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
__device__ constexpr int vmcnt_only(int n)
{
    return (n & 0xF) | (0x7 << 4) | (0xF << 8) | ((n >> 4) << 14);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes)
{
    // dword3 0x00020000: 32-bit untyped data format, no swizzle (gfx9 family)
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             0x00020000);
}

// Direct loads: load p of wave w fills the 1 KiB LDS block 4p + w of a tile;
// lane L writes its bytes 16L..16L+15, which hold (row, chunk) with
// chunk = physical chunk ^ swizzle(row). Rows of load p are those of load 0
// plus p * ROWS_PER_LOAD, and the swizzle only sees the row modulo 16, so the
// per-lane byte offset is the same for every p and every tile; the tile's
// and the load's row steps are a wave-uniform addend.
template <class T>
__device__ __forceinline__ uint32_t load_lane_offset(int wave, int lane, int64_t stride)
{
    int pos = wave * 1024 + 16 * lane;
    int row = pos / T::ROWB;
    int pc = (pos % T::ROWB) / 16;
    int c = pc ^ chunk_swizzle<T::D>(row);
    return (uint32_t)(((int64_t)row * stride + 8 * c) * 2);
}

// Issue the direct global->LDS loads of one tile: rows j0..j0+BN-1 of the
// slice described by `rs` (whose range ends at the sequence end, so rows past
// it read as zero). The row offset is wave-uniform and added to the lane's
// constant byte offset. (Advancing the descriptor's base by the row offset
// instead, as scalar work, measured 1-2.5 % slower: seven scalar
// instructions per load in the wave's in-order stream against one vector
// add.)
template <class T>
__device__ __forceinline__ void issue_load(char* lds_tile, __amdgpu_buffer_rsrc_t rs, int j0,
                                           uint32_t row_bytes, uint32_t lane_off, int wave, int p)
{
    const uint32_t off = lane_off + (uint32_t)(j0 + p * T::ROWS_PER_LOAD) * row_bytes;
    // Soft-cap and left-bounded softmax kernels: an opaque wave offset makes
    // each load form its LDS address from one register, where the compiler
    // would otherwise keep one hoisted address per load and buffer, spill
    // them from the scalar registers and reload them into the loop with
    // vector instructions.
    int wo = wave * 1024;
    if constexpr (T::CAP != kCapOff || (T::LEFT && T::SOFTMAX)) asm volatile("" : "+s"(wo));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (lds_void*)(lds_tile + 4096 * p + wo), 16, off, 0, 0, 0);
}

// All LOADS loads of this wave for one tile.
template <class T>
__device__ __forceinline__ void issue_tile(char* lds_tile, __amdgpu_buffer_rsrc_t rs, int j0,
                                           uint32_t row_bytes, uint32_t lane_off, int wave)
{
#pragma unroll
    for (int p = 0; p < T::LOADS; ++p) issue_load<T>(lds_tile, rs, j0, row_bytes, lane_off, wave, p);
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b)
{
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 v;
    v[0] = (__bf16)a;
    v[1] = (__bf16)b;
    return __builtin_bit_cast(uint32_t, v);
}

// a + b of the bf16 pair packed in `w`, added to `acc` (one dot product
// with (1, 1); the products are exact).
__device__ __forceinline__ float add_bf16_pair(uint32_t w, float acc)
{
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, acc, false);
}

// Lanes l and l ^ 32 hold the two halves of the same query row.
__device__ __forceinline__ float pair_max(float x)
{
    auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                              __builtin_bit_cast(uint32_t, x), false, false);
    return __builtin_fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]),
                           __builtin_bit_cast(float, (uint32_t)r[1]));
}

__device__ __forceinline__ float pair_sum(float x)
{
    auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                              __builtin_bit_cast(uint32_t, x), false, false);
    return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

// Sequence, first query head of the workgroup's head set, kv head, query
// tile; qt < 0: no work item (past the end of a packed grid).
struct WorkItem {
    int b, hq, hkv, qt;
};

// Compile-time loop: f(std::integral_constant<int, i>) for i = 0..N-1, so
// every index is a constant and per-iteration arrays stay in registers.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}

template <int N, class F>
__device__ __forceinline__ void static_for(F&& f)
{
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int V>
struct Parity {
    static constexpr int value = V;
};

template <bool V>
struct Bool {
    static constexpr bool value = V;
};

// Map the hardware workgroup id to (sequence, query head set, query tile).
// Query tiles are issued longest-first: the last tiles of a causal sequence
// see the most keys, so the order is descending unless the host asks for
// ascending (q_order = 1: the first tiles are the heaviest, e.g. global rows).
// With hp heads per workgroup (32 * 4 / hp rows), the hp query tiles of one
// 128-row span of a head set have consecutive ids, so they start together
// on one XCD and read the same K/V tiles at about the same time.
// Mode 1 keeps all query heads of a kv-head group on one XCD (workgroup ids
// are dealt round-robin over the 8 XCDs), so their K/V tiles are shared
// through that XCD's L2. Within an XCD the kv-head groups are taken `chunk`
// at a time (every head set and query tile of the chunk, longest-first
// inside it), so the K/V tiles in use at any moment belong to a few groups
// and stay in the L2 instead of cycling every group's K/V through the
// caches once per tile.
// Packed variable-length grid (compact, with mode 1 and one kv group per
// chunk): an XCD's work items are those of its groups g = x + 8 i in order i,
// each group contributing only the query tiles of its own sequence
// (ceil(length / tile rows) tiles, times its head sets), in the order of the
// padded grid (128-row spans of hp tiles, the last span holding only the
// tiles that have rows), so no workgroup is spent on tiles past a
// sequence's end. Every wave finds its group from the prefix
// sums of the item counts over the XCD's groups, 256 groups at a time (four
// consecutive groups per lane, their length loads issued together, so a batch
// of thousands of sequences waits on a quarter of the load round trips).
__device__ __forceinline__ WorkItem decode_packed(const AttnParams& p, uint32_t uw)
{
    constexpr int PER = 4;  // groups per lane and round
    WorkItem it = {0, 0, 0, -1};
    const uint32_t x = uw & 7, k = uw >> 3;
    const int lane = __lane_id();
    uint32_t base = 0;  // items of the groups before this round's 256
    for (int i0 = 0; i0 < p.groups_per_xcd; i0 += 64 * PER) {
        uint32_t n[PER], b[PER], tiles[PER];
        uint32_t sum = 0;
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int i = i0 + PER * lane + u;
            n[u] = 0;
            b[u] = 0;
            tiles[u] = 0;
            if (i < p.groups_per_xcd) {
                b[u] = fast_div(x + 8u * (uint32_t)i, p.div_hkv);
                const int len = p.cu_q[b[u] + 1] - p.cu_q[b[u]];
                // tiles of 128 / hp rows
                tiles[u] = (uint32_t)(len + (127 >> p.hp_shift)) >> (7 - p.hp_shift);
                n[u] = tiles[u] * (uint32_t)p.items_per_tile;
            }
            sum += n[u];
        }
        uint32_t incl = sum;  // inclusive prefix sum over the lanes
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t t = (uint32_t)__shfl_up((int)incl, d);
            if (lane >= d) incl += t;
        }
        const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
        if (k < base + total) {
            // the first lane whose groups reach past item k holds its group
            const uint64_t hit = __builtin_amdgcn_ballot_w64(base + incl > k);
            const int j = __builtin_ctzll(hit);
            uint32_t before =
                base + __builtin_amdgcn_readlane(incl, j) - __builtin_amdgcn_readlane(sum, j);
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                const uint32_t nu = __builtin_amdgcn_readlane(n[u], j);
                if (k < before + nu) {
                    const uint32_t rem = k - before;
                    const uint32_t g = x + 8u * (uint32_t)(i0 + PER * j + u);
                    const uint32_t bj = __builtin_amdgcn_readlane(b[u], j);
                    const uint32_t nt = __builtin_amdgcn_readlane(tiles[u], j);
                    // inside the group: 128-row spans of hp tiles (the last
                    // one holding t_top tiles), each span's items ordered by
                    // head set, then tile; spans from the top (q_order 0) or
                    // from the bottom (q_order 1), as in the padded grid
                    const uint32_t hpu = (uint32_t)p.hp, gsets = p.div_group.d;
                    const uint32_t sj = (nt + hpu - 1) >> p.hp_shift;       // spans, >= 1
                    const uint32_t t_top = nt - ((sj - 1) << p.hp_shift);  // 1 .. hp
                    const uint32_t top_first = p.q_order ? 0u : t_top * gsets;
                    const uint32_t top_lo = p.q_order ? (sj - 1) * hpu * gsets : 0u;
                    uint32_t r, qt;
                    if (rem >= top_lo && rem < top_lo + t_top * gsets) {  // the last span
                        const uint32_t e = rem - top_lo;
                        r = e / t_top;
                        const uint32_t lo = e - r * t_top;
                        qt = ((sj - 1) << p.hp_shift) + (p.q_order ? lo : t_top - 1 - lo);
                    } else {  // a full span
                        const uint32_t e = rem - top_first;
                        const uint32_t lo = e & (hpu - 1), rest = e >> p.hp_shift;
                        const uint32_t hi = fast_div(rest, p.div_group);
                        r = rest - hi * gsets;
                        qt = p.q_order ? (hi << p.hp_shift) + lo
                                       : ((sj - 2 - hi) << p.hp_shift) + (hpu - 1 - lo);
                    }
                    it.b = (int)bj;
                    it.hkv = (int)(g - bj * p.div_hkv.d);
                    it.hq = it.hkv * p.group + (int)(r << p.hp_shift);
                    it.qt = (int)qt;
                    return it;
                }
                before += nu;
            }
        }
        base += total;
    }
    return it;
}

__device__ __forceinline__ WorkItem decode_block(const AttnParams& p, int w)
{
    // every divisor is launch-invariant: multiply-high and shift (fastdiv.h)
    WorkItem it;
    const uint32_t uw = (uint32_t)w;
    int qt_rev;
    if (p.compact) return decode_packed(p, uw);
    if (p.map_mode == 1) {
        const uint32_t x = uw & 7, k = uw >> 3;
        const uint32_t c = fast_div(k, p.div_chunk_items);
        const uint32_t rem = k - c * p.div_chunk_items.d;
        const uint32_t lo = rem & (uint32_t)(p.hp - 1), rest = rem >> p.hp_shift;
        // (head set in group, group in chunk) pairs of this chunk
        const FastDiv pairs = (int)c == p.last_chunk ? p.div_chunk_last : p.div_chunk_full;
        const uint32_t hi = fast_div(rest, pairs);
        qt_rev = (int)((hi << p.hp_shift) + lo);
        const uint32_t r2 = rest - hi * pairs.d;
        const uint32_t gq = fast_div(r2, p.div_group);
        const int r = (int)(r2 - gq * p.div_group.d);  // head set within the group
        const uint32_t g = x + 8 * (c * (uint32_t)p.chunk + gq);
        const uint32_t b = fast_div(g, p.div_hkv);
        it.b = (int)b;
        it.hkv = (int)(g - b * p.div_hkv.d);
        it.hq = it.hkv * p.group + (r << p.hp_shift);
    } else {
        const uint32_t lo = uw & (uint32_t)(p.hp - 1), rest = uw >> p.hp_shift;
        const uint32_t hi = fast_div(rest, p.div_bh);
        qt_rev = (int)((hi << p.hp_shift) + lo);
        const uint32_t rem = rest - hi * p.div_bh.d;
        const uint32_t b = fast_div(rem, p.div_hq);
        const uint32_t hs = rem - b * p.div_hq.d;  // head set
        it.b = (int)b;
        it.hq = (int)(hs << p.hp_shift);
        it.hkv = (int)fast_div(hs, p.div_group);
    }
    it.qt = p.q_order ? qt_rev : p.num_q_tiles - 1 - qt_rev;
    return it;
}

// Per-wavefront state carried through the key loop.
template <class T>
struct WaveState {
    bf16x8 qf[T::KSTEPS];      // Q fragment (B operand of S^T)
    int kaddr[T::KSTEPS];      // LDS byte offsets of this lane's K reads
    int vaddr[T::DBLK][2];     // LDS byte offsets of this lane's V transpose reads
    f32x16 oacc[T::DBLK];      // O^T accumulator
    f32x16 sa[T::NB], sb[T::NB];  // scores of tiles of even / odd parity
    float m_run, l_run;           // softmax only: running max (units) and partial row sum
    float l_o;                    // softmax only: partial row sum of P as rounded to bf16
    float alpha;                  // softmax with mods: rescale factor of O and l
    bool need;                    // softmax with mods: O and l must be rescaled
    // row constants: visible keys j < pfx (general path) and jlo <= j <= jhi;
    // key-axis position ip; relative-position reference jref
    int lh, pfx, jlo, jhi, ip, jref;
    float bias_abs, bias_lin;  // coefficients of |ip - j| and (jref - j), in units
};

// Visible-key bounds of this lane's row relative to the key of element
// offset 0 in a tile (jn + 8 lh), so each element compares its compile-time
// offset c = 32b + e + (e >= 8 ? 8 : 0) directly.
struct MaskThr {
    int lo, hi, pf;
};

template <class T>
__device__ __forceinline__ MaskThr mask_thresholds(const WaveState<T>& ws, int jn)
{
    const int base = jn + 8 * ws.lh;
    return {ws.jlo - base, ws.jhi - base, ws.pfx - base};
}

template <class T>
__device__ __forceinline__ bool visible(const MaskThr& m, int c)
{
    if constexpr (T::GEN)
        return c < m.pf || (c >= m.lo && c <= m.hi);
    else if constexpr (T::LEFT)
        return c >= m.lo && c <= m.hi;
    else
        return c <= m.hi;
}

// Per-tile bases of the position terms of this lane's row: with j the key
// at element offset 0 of the lane (jn + 8 lh), i' - j and jref - j as floats;
// an element at offset c then takes base - c.
struct PosBase {
    float abs, lin;
};

template <class T>
__device__ __forceinline__ PosBase pos_base(const WaveState<T>& ws, int jn)
{
    if constexpr (T::BIAS == kBiasNone) return {0.0f, 0.0f};
    const int j = jn + 8 * ws.lh;
    return {(float)(ws.ip - j), (float)(ws.jref - j)};
}

// Final score of element offset c (units; see score_tile_u).
template <class T>
__device__ __forceinline__ float final_score(float x, const AttnParams& p, const WaveState<T>& ws,
                                             const PosBase& pb, int c)
{
    return score_tile_u<T::CAP, T::BIAS>(x, p.scale_u,
                                         T::CAP == kCapShort ? p.softcap_pre2 : p.softcap_pre,
                                         p.softcap_post_u,
                                              ws.bias_abs, ws.bias_lin, pb.abs - (float)c,
                                              pb.lin - (float)c);
}

// Side of a key tile relative to every row of the workgroup (DIAG): all its
// keys at or before every row's key-axis position, all at or after, or
// neither (or not known).
enum : int { kSideBoth = 0, kSideLeft = 1, kSideRight = 2 };

// FOLD: this lane's additive constant of a tile's scores: the short soft-cap
// form's C' (it ends in C' - 2C'/(1 + e); not with POLY, whose polynomial
// carries no constant), minus the running max m_base, plus the per-tile part
// of the position terms (ALiBi on one-sided tiles, the relative position term
// always).
template <class T, int SIDE>
__device__ __forceinline__ float fold_const(const WaveState<T>& ws, const AttnParams& p,
                                            const PosBase& pb, float m_base)
{
    float a = (T::CAP == kCapShort && !T::POLY ? p.softcap_post_u : 0.0f) - m_base;
    if constexpr (T::BIAS == kBiasAlibi && SIDE == kSideLeft) a = __builtin_fmaf(ws.bias_abs, pb.abs, a);
    if constexpr (T::BIAS == kBiasAlibi && SIDE == kSideRight) a = __builtin_fmaf(-ws.bias_abs, pb.abs, a);
    if constexpr (T::BIAS == kBiasRelPos) a = __builtin_fmaf(ws.bias_lin, pb.lin, a);
    return a;
}

// FOLD: the final score of element offset c minus the running max, from the
// raw dot product and the tile constant a of fold_const. With POLY the
// soft-cap is C' tanh(y) = dot (b0 + z (b1 + z b2)), z = dot^2, an odd
// polynomial valid while z <= cap_zmax (|y| <= R, the range the host chose
// for C so that the score errs by at most 1e-4 units; softcap_poly.h), three
// plain operations where the short form takes two transcendental ones; EXACT
// (the fallback of a tile with a larger |y|) takes the short form and adds
// the C' that a then lacks.
template <class T, int SIDE, bool EXACT = false>
__device__ __forceinline__ float fold_score(float dot, float z, float a, const AttnParams& p,
                                            const WaveState<T>& ws, const PosBase& pb, int c)
{
    float u;
    if constexpr (T::POLY && !EXACT) {
        float q = __builtin_fmaf(z, p.cap_poly[2], p.cap_poly[1]);
        q = __builtin_fmaf(z, q, p.cap_poly[0]);
        u = __builtin_fmaf(dot, q, a);
    } else if constexpr (T::POLY) {
        const float e = __builtin_amdgcn_exp2f(dot * p.softcap_pre2);
        u = __builtin_fmaf(-2.0f * p.softcap_post_u, __builtin_amdgcn_rcpf(1.0f + e),
                           a + p.softcap_post_u);
    } else if constexpr (T::CAP == kCapShort) {
        const float e = __builtin_amdgcn_exp2f(dot * p.softcap_pre2);
        u = __builtin_fmaf(-2.0f * p.softcap_post_u, __builtin_amdgcn_rcpf(1.0f + e), a);
    } else if constexpr (T::CAP == kCapExact) {
        u = softcap_u(dot, p.softcap_pre, p.softcap_post_u) + a;
    } else {
        u = __builtin_fmaf(dot, p.scale_u, a);
    }
    if constexpr (T::BIAS == kBiasAlibi) {
        if constexpr (SIDE == kSideLeft)  // |i' - j| = base - c
            u = __builtin_fmaf((float)c, -ws.bias_abs, u);
        else if constexpr (SIDE == kSideRight)  // |i' - j| = c - base
            u = __builtin_fmaf((float)c, ws.bias_abs, u);
        else
            u = __builtin_fmaf(ws.bias_abs, __builtin_fabsf(pb.abs - (float)c), u);
    }
    if constexpr (T::BIAS == kBiasRelPos) u = __builtin_fmaf((float)c, -ws.bias_lin, u);
    return u;
}

// S^T = K Q^T for the K tile in LDS at `kt`.
template <class T>
__device__ __forceinline__ void qk_tile(const char* kt, const WaveState<T>& ws, f32x16 (&s)[T::NB])
{
#pragma unroll
    for (int b = 0; b < T::NB; ++b) {
#pragma unroll
        for (int t = 0; t < T::KSTEPS; ++t) {
            bf16x8 a = *reinterpret_cast<const bf16x8*>(kt + 32 * b * T::ROWB + ws.kaddr[t]);
            s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, ws.qf[t], t == 0 ? f32x16{} : s[b], 0,
                                                           0, 0);
        }
    }
    // Issue order: K reads AHEAD products ahead, then one product and one read
    // at a time, block by block (each accumulation chain back to back: faster
    // than the compiler's own interleaving of the two chains).
    constexpr int N = T::NB * T::KSTEPS, AHEAD = 4;
    __builtin_amdgcn_sched_group_barrier(0x100, AHEAD, 0);  // DS read
#pragma unroll
    for (int i = 0; i < N - AHEAD; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, AHEAD, 0);
}

// Score mods, element mask (MASKED) and the tile's row max, in log2 units.
template <class T, bool MASKED>
__device__ __forceinline__ float mods_and_max(f32x16 (&s)[T::NB], const AttnParams& p,
                                              const WaveState<T>& ws, int j0)
{
    float mx = -__builtin_inff();
    const MaskThr mt = mask_thresholds(ws, j0);
    const PosBase pb = pos_base(ws, j0);
#pragma unroll
    for (int b = 0; b < T::NB; ++b) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            // element (b, e) is key j0 + 8lh + c, c = 32b + e + (e >= 8 ? 8 : 0)
            const int c = 32 * b + e + (e >= 8 ? 8 : 0);
            float x = s[b][e];
            if constexpr (T::MODS) x = final_score<T>(x, p, ws, pb, c);
            if constexpr (MASKED)
                if (!visible<T>(mt, c)) x = -__builtin_inff();
            s[b][e] = x;
            mx = __builtin_fmaxf(mx, x);
        }
    }
    if constexpr (!T::SOFTMAX) return 0.0f;
    mx = pair_max(mx);
    if constexpr (!T::MODS) mx *= p.scale_u;  // raw max -> log2 units (scale > 0)
    return mx;
}

// Norm of one score (in units; raw dot product when there are no mods):
// softmax exp2(S - m), or the ReLU / Sigmoid activation of the natural score.
// SHIFT = false (FOLD): the score already has the running max taken off.
template <class T, bool SHIFT = true>
__device__ __forceinline__ float norm_value(float x, float m_use, float scale_u)
{
    if constexpr (T::SOFTMAX) {
        if constexpr (T::FOLD && !SHIFT) return __builtin_amdgcn_exp2f(x);
        return __builtin_amdgcn_exp2f(T::MODS ? x - m_use : __builtin_fmaf(x, scale_u, -m_use));
    } else {
        return activation<T::NORM>(T::MODS ? x : x * scale_u);
    }
}

// Softmax with mods: fold a tile max into the running max; decide whether O
// must be rescaled (only when the max grew by more than TAU).
template <class T>
__device__ __forceinline__ void update_max(WaveState<T>& ws, float mx)
{
    if constexpr (!T::SOFTMAX || T::MAXFREE) return;
    const float m_new = __builtin_fmaxf(ws.m_run, mx);
    ws.need = m_new > ws.m_run + TAU;
    ws.alpha = ws.need ? __builtin_amdgcn_exp2f(ws.m_run - m_new) : 1.0f;
    if (ws.need) ws.m_run = m_new;
}

template <class T>
__device__ __forceinline__ void rescale_if_needed(WaveState<T>& ws)
{
    if constexpr (!T::SOFTMAX || T::MAXFREE) return;
    if (__builtin_amdgcn_ballot_w64(ws.need)) {
        ws.l_run *= ws.alpha;
        ws.l_o *= ws.alpha;
#pragma unroll
        for (int d = 0; d < T::DBLK; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) ws.oacc[d][e] *= ws.alpha;
    }
}

// Does the row of this lane see a key of the tile starting at key jc?
template <class T>
__device__ __forceinline__ bool row_sees_tile(const WaveState<T>& ws, int jc)
{
    const bool band = ws.jlo <= ws.jhi && ws.jlo <= jc + T::BN - 1 && ws.jhi >= jc;
    if constexpr (T::GEN) return band || ws.pfx > jc;
    return band;
}

// This lane's partial row sums of a tile's P: f in fp32 (the softmax
// denominator) and, with PSUM_BF16, b of P as rounded to bf16, the values the
// P V product multiplies, which then normalises O. With the running max
// behind the row max (lazily updated, or not at all on the check-free path),
// the largest P of a row is not 1, and its bf16 rounding error (up to 2^-8
// relative) passes into O unmatched by an fp32 denominator: visible in rows
// that see few keys.
struct RowSums {
    float f, b;
};

// P = Norm(S) as bf16 B operands of the P V product; returns (softmax) this
// lane's partial row sums.
template <class T, bool SHIFT = true>
__device__ __forceinline__ RowSums exp_tile(const f32x16 (&s)[T::NB], u32x4 (&pw)[T::NB][2],
                                            float m_use, float scale_u)
{
    RowSums rs = {-0.0f, -0.0f};  // -0 + x == x for every x: the first add folds away
#pragma unroll
    for (int b = 0; b < T::NB; ++b) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float p0 = norm_value<T, SHIFT>(s[b][8 * u + 2 * q], m_use, scale_u);
                float p1 = norm_value<T, SHIFT>(s[b][8 * u + 2 * q + 1], m_use, scale_u);
                pw[b][u][q] = pack_bf16(p0, p1);
                if constexpr (T::SOFTMAX) {
                    rs.f += p0;
                    rs.f += p1;
                }
                if constexpr (T::PSUM_BF16) rs.b = add_bf16_pair(pw[b][u][q], rs.b);
            }
        }
    }
    return rs;
}

// After the exponentials of tile j (first key jc) the row sums join l. With
// MAXFREE the exponentials were made with the running max as it stands (0
// while a row has seen no key): P is kept when every lane's partial sum stays
// within PSUM_BOUND and no row sees its first keys in this tile. Otherwise
// (rare: the first keys of a row whose first tile this is not, a jump of the
// max) the running max of the affected rows moves to the max over the tile's
// scores, O and l are rescaled, and P and the row sums are recomputed from
// the scores. The two lanes of a row take the same decision. The row max
// then plays no part in the common path, which saves its reductions on every
// tile.
template <class T>
__device__ __forceinline__ void check_tile(WaveState<T>& ws, const f32x16 (&s)[T::NB],
                                           u32x4 (&pw)[T::NB][2], RowSums rs, const AttnParams& p,
                                           int jc)
{
    if constexpr (!T::SOFTMAX) return;
    if constexpr (!T::MAXFREE) {
        ws.l_run += rs.f;
        if constexpr (T::PSUM_BF16) ws.l_o += rs.b;
        return;
    }
    bool need = rs.f > PSUM_BOUND;
    if (ws.m_run == -__builtin_inff()) need = need || row_sees_tile(ws, jc);
    if (__builtin_amdgcn_ballot_w64(need)) {
        const bool need_row = pair_max(need ? 1.0f : 0.0f) > 0.0f;
        float tm = -__builtin_inff();
#pragma unroll
        for (int b = 0; b < T::NB; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) tm = __builtin_fmaxf(tm, s[b][e]);
        tm = pair_max(tm);
        if constexpr (!T::MODS) tm *= p.scale_u;  // raw max -> units (scale > 0)
        const float m_old = ws.m_run;
        // FOLD: the scores carry -m_old (-0 while the row has seen no key)
        const float m_base = T::FOLD && m_old != -__builtin_inff() ? m_old : 0.0f;
        if constexpr (T::FOLD) tm += m_base;
        const float m_new = need_row ? __builtin_fmaxf(m_old, tm) : m_old;
        const float alpha =
            need_row && m_old != -__builtin_inff() ? __builtin_amdgcn_exp2f(m_old - m_new) : 1.0f;
        ws.m_run = m_new;
        ws.l_run *= alpha;
        ws.l_o *= alpha;
#pragma unroll
        for (int d = 0; d < T::DBLK; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) ws.oacc[d][e] *= alpha;
        rs = exp_tile<T, true>(s, pw, (m_new == -__builtin_inff() ? 0.0f : m_new) - m_base,
                               p.scale_u);
    }
    ws.l_run += rs.f;
    if constexpr (T::PSUM_BF16) ws.l_o += rs.b;
}

// O^T += V^T P^T for the V tile in LDS at `vt`.
template <class T>
__device__ __forceinline__ void pv_tile(const char* vt, const u32x4 (&pw)[T::NB][2], WaveState<T>& ws)
{
#pragma unroll
    for (int b = 0; b < T::NB; ++b) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            bf16x8 pb = __builtin_bit_cast(bf16x8, pw[b][u]);
            const int kb = (32 * b + 16 * u) * T::ROWB;
#pragma unroll
            for (int d = 0; d < T::DBLK; ++d) {
                s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4*)(vt + kb + ws.vaddr[d][0]));
                s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_s16x4*)(vt + kb + ws.vaddr[d][1]));
                s16x8 a8 = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                ws.oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a8), pb, ws.oacc[d], 0, 0, 0);
            }
        }
    }
}

// One pipelined step, written out as explicit slices. Each QK^T slice issues
// one MFMA of S_next = Q K_next^T, the K read of the MFMA PF slices later, an
// equal share of the exponentials of the current tile (P and row sum) and,
// in the first slices, one of the global->LDS loads of the tiles the next
// step reads (`load(i)`, i < 2 LOADS), whose issue then overlaps the matrix
// products; each P V slice issues one MFMA of O^T += V^T P^T, the two
// transpose reads of a later MFMA and a share of the score mods, mask and max
// of S_next. A scheduling barrier after every slice keeps this order, so the
// vector work runs while the matrix cores are busy and LDS latency stays
// hidden. The QK^T products run block by block, each accumulation chain
// issued back to back, the order that measured fastest.
template <class T, bool MASKED, int SIDE, class LOADER>
__device__ __forceinline__ void pipelined_step(const char* kread, const char* vread,
                                               WaveState<T>& ws, const f32x16 (&sc)[T::NB],
                                               f32x16 (&sn)[T::NB], const AttnParams& p,
                                               float m_use, int jc, int jn, LOADER&& load)
{
    constexpr int NB = T::NB, DBLK = T::DBLK;
    constexpr int QK = T::KSTEPS * NB;   // QK^T MFMAs (block-major, k-step-minor)
    constexpr int NLD = 2 * T::LOADS;    // loads of the next step's K and V tiles
    constexpr int LSTEP = QK / NLD;      // one load every LSTEP slices
    static_assert(LSTEP >= 1 && LSTEP * NLD == QK, "load split");
    constexpr int PV = 2 * NB * DBLK;    // P V MFMAs (b, u, d)
    constexpr int PF = 3;                // read prefetch distance in slices
    constexpr int EQ = 16 * NB / QK;     // exponentials per QK slice
    constexpr int EP = 16 * NB / PV;     // score elements per P V slice
    static_assert(EQ % 2 == 0 && EQ * QK == 16 * NB && EP * PV == 16 * NB, "slice split");

    u32x4 pw[NB][2];
    bf16x8 kop[QK];
    s16x4 vlo[PV], vhi[PV];
    RowSums rs = {-0.0f, -0.0f};  // -0 + x == x for every x: the first add folds away
    float mx = -__builtin_inff();
    float zmax = 0.0f;  // POLY: the largest dot^2 of the next tile

    auto read_k = [&](int i) __attribute__((always_inline)) {
        const int b = i / T::KSTEPS, t = i % T::KSTEPS;
        kop[i] = *reinterpret_cast<const bf16x8*>(kread + 32 * b * T::ROWB + ws.kaddr[t]);
    };
    auto read_v = [&](int i) __attribute__((always_inline)) {
        const int b = i / (2 * DBLK), u = (i / DBLK) % 2, d = i % DBLK;
        const int kb = (32 * b + 16 * u) * T::ROWB;
        vlo[i] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vread + kb + ws.vaddr[d][0]));
        vhi[i] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vread + kb + ws.vaddr[d][1]));
    };

    static_for<PF>([&](auto ic) __attribute__((always_inline)) { read_k(ic.value); });
    __builtin_amdgcn_sched_barrier(0);
    static_for<QK>([&](auto ic) __attribute__((always_inline)) {
        constexpr int i = ic.value, b = i / T::KSTEPS, t = i % T::KSTEPS;
        if constexpr (t == 0)
            sn[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[i], ws.qf[t], f32x16{}, 0, 0, 0);
        else
            sn[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[i], ws.qf[t], sn[b], 0, 0, 0);
        if constexpr (i + PF < QK)
            read_k(i + PF);
        else
            read_v(i + PF - QK);
        if constexpr (i % LSTEP == 0) load(i / LSTEP);
        static_for<EQ / 2>([&](auto kc) __attribute__((always_inline)) {
            constexpr int el = i * EQ + 2 * kc.value, bb = el / 16, e = el % 16;
            const float p0 = norm_value<T, !T::FOLD>(sc[bb][e], m_use, p.scale_u);
            const float p1 = norm_value<T, !T::FOLD>(sc[bb][e + 1], m_use, p.scale_u);
            pw[bb][e / 8][(e % 8) / 2] = pack_bf16(p0, p1);
            // MAXFREE: keep the conversion in this slice. check_tile may
            // recompute P, so the compiler would otherwise sink it past the
            // check, where it runs unhidden before the first P V product and
            // keeps the fp32 P alive across the branch.
            if constexpr (T::MAXFREE) asm volatile("" : "+v"(pw[bb][e / 8][(e % 8) / 2]));
            if constexpr (T::SOFTMAX) {
                rs.f += p0;
                rs.f += p1;
            }
            if constexpr (T::PSUM_BF16) rs.b = add_bf16_pair(pw[bb][e / 8][(e % 8) / 2], rs.b);
        });
        __builtin_amdgcn_sched_barrier(0);
    });
    check_tile<T>(ws, sc, pw, rs, p, jc);
    const MaskThr mt = mask_thresholds(ws, jn);
    const PosBase pb = pos_base(ws, jn);
    // FOLD: the next tile's scores take off the running max as it now stands
    float fa = 0.0f;
    if constexpr (T::FOLD)
        fa = fold_const<T, SIDE>(ws, p, pb, ws.m_run == -__builtin_inff() ? 0.0f : ws.m_run);
    static_for<PV>([&](auto ic) __attribute__((always_inline)) {
        constexpr int i = ic.value;
        constexpr int b = i / (2 * DBLK), u = (i / DBLK) % 2, d = i % DBLK;
        s16x8 a8 = __builtin_shufflevector(vlo[i], vhi[i], 0, 1, 2, 3, 4, 5, 6, 7);
        ws.oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a8),
                                                             __builtin_bit_cast(bf16x8, pw[b][u]),
                                                             ws.oacc[d], 0, 0, 0);
        if constexpr (i + PF < PV) read_v(i + PF);
        static_for<EP>([&](auto kc) __attribute__((always_inline)) {
            constexpr int el = i * EP + kc.value, bb = el / 16, e = el % 16;
            // element (bb, e) is key jn + 8lh + c, c = 32bb + e + (e >= 8 ? 8 : 0)
            constexpr int c = 32 * bb + e + (e >= 8 ? 8 : 0);
            float x = sn[bb][e];
            if constexpr (T::POLY) {
                const float z = x * x;
                zmax = __builtin_fmaxf(zmax, z);
                x = fold_score<T, SIDE>(x, z, fa, p, ws, pb, c);
                // keep the score's arithmetic in this slice: the fallback below
                // overwrites it, so the compiler would otherwise sink it past
                // the products into the common path's successor
                asm volatile("" : "+v"(x));
            } else if constexpr (T::FOLD)
                x = fold_score<T, SIDE>(x, 0.0f, fa, p, ws, pb, c);
            else if constexpr (T::MODS)
                x = final_score<T>(x, p, ws, pb, c);
            if constexpr (MASKED)
                if (!visible<T>(mt, c)) x = -__builtin_inff();
            sn[bb][e] = x;
            if constexpr (T::SOFTMAX && !T::MAXFREE) mx = __builtin_fmaxf(mx, x);
        });
        __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (T::SOFTMAX && !T::MAXFREE) {
        mx = pair_max(mx);
        if constexpr (!T::MODS) mx *= p.scale_u;  // raw max -> log2 units (scale > 0)
        update_max(ws, mx);
    }
    if constexpr (T::POLY) {
        // Rare: a score of the tile lies beyond the polynomial's range. K of
        // the tile is still in LDS (the next step's loads fill the other
        // buffer), so the wave recomputes its dot products and takes the
        // short form for the whole tile.
        if (__builtin_amdgcn_ballot_w64(zmax > p.cap_zmax)) {
            qk_tile<T>(kread, ws, sn);
#pragma unroll
            for (int bb = 0; bb < NB; ++bb)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int c = 32 * bb + e + (e >= 8 ? 8 : 0);
                    float x = fold_score<T, SIDE, true>(sn[bb][e], 0.0f, fa, p, ws, pb, c);
                    if constexpr (MASKED)
                        if (!visible<T>(mt, c)) x = -__builtin_inff();
                    sn[bb][e] = x;
                }
        }
    }
}

// The last step of the key loop: exponentials and P V of the current tile.
template <class T>
__device__ __forceinline__ void last_step(const char* vread, WaveState<T>& ws, f32x16 (&sc)[T::NB],
                                          const AttnParams& p, float m_use, int jc)
{
    // No row of this wave sees the tile (the diagonal tile of the upper rows
    // under causal-like masks): P is zero, nothing to add.
    if (!__builtin_amdgcn_ballot_w64(row_sees_tile(ws, jc))) return;
    u32x4 pw[T::NB][2];
    const RowSums rs = exp_tile<T, !T::FOLD>(sc, pw, m_use, p.scale_u);
    check_tile<T>(ws, sc, pw, rs, p, jc);
    pv_tile<T>(vread, pw, ws);
}

// Keys of a listed global set G that a row does not already see through its
// band (Appendix A, Global Sliding Window: j in G is visible from every row),
// visited after the planned tiles, BN list entries at a time. `gl` holds G in
// LDS, sorted and padded with lk (past the sequence end) to a multiple of BN.
// The K and V rows of such a gathered tile are fetched one by one (each lane's
// direct loads take the row of its list entry) into the first K/V buffers in
// the usual swizzled layout, and every element is masked and modified with its
// own key position; the online softmax state simply continues.
template <class T>
__device__ void gathered_tiles(WaveState<T>& ws, const AttnParams& p, const int* gl, int ng,
                               char* lds_k, char* lds_v, __amdgpu_buffer_rsrc_t krs,
                               __amdgpu_buffer_rsrc_t vrs, uint32_t krow, uint32_t vrow, int lk,
                               bool row_valid, int wave, int lane)
{
    // tile row and swizzled 16-byte chunk this lane loads in load 0 (load q
    // covers the rows q * ROWS_PER_LOAD further, whose swizzle is the same)
    const int pos0 = wave * 1024 + 16 * lane;
    const int r0 = pos0 / T::ROWB;
    const uint32_t chunk = (uint32_t)((((pos0 % T::ROWB) / 16) ^ chunk_swizzle<T::D>(r0)) * 16);
    for (int g0 = 0; g0 < ng; g0 += T::BN) {
        __syncthreads();  // every wave is done with the buffers
#pragma unroll
        for (int q = 0; q < T::LOADS; ++q) {
            // rows past the sequence end (padding, or positions >= lk) read as zero
            const int key = min(gl[g0 + r0 + q * T::ROWS_PER_LOAD], lk);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                krs, (lds_void*)(lds_k + (4 * q + wave) * 1024), 16, chunk + (uint32_t)key * krow, 0,
                0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                vrs, (lds_void*)(lds_v + (4 * q + wave) * 1024), 16, chunk + (uint32_t)key * vrow, 0,
                0, 0);
        }
        __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
        __syncthreads();
        qk_tile<T>(lds_k, ws, ws.sa);
        float mx = -__builtin_inff();
#pragma unroll
        for (int b = 0; b < T::NB; ++b) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                // element (b, e) is list entry g0 + 8 lh + c
                const int c = 32 * b + e + (e >= 8 ? 8 : 0);
                const int j = gl[g0 + 8 * ws.lh + c];
                float x = ws.sa[b][e];
                if constexpr (T::MODS)
                    x = score_tile_u<T::CAP, T::BIAS>(
                        x, p.scale_u, T::CAP == kCapShort ? p.softcap_pre2 : p.softcap_pre,
                        p.softcap_post_u, ws.bias_abs, ws.bias_lin, (float)(ws.ip - j),
                        (float)(ws.jref - j));
                const bool vis = row_valid && j < lk && !(j >= ws.jlo && j <= ws.jhi);
                x = vis ? x : -__builtin_inff();
                ws.sa[b][e] = x;
                mx = __builtin_fmaxf(mx, x);
            }
        }
        if constexpr (T::SOFTMAX) {
            mx = pair_max(mx);
            if constexpr (!T::MODS) mx *= p.scale_u;  // raw max -> units (scale > 0)
            update_max(ws, mx);
            rescale_if_needed(ws);
        }
        const float m_use = ws.m_run == -__builtin_inff() ? 0.0f : ws.m_run;
        u32x4 pw[T::NB][2];
        const RowSums rs = exp_tile<T>(ws.sa, pw, m_use, p.scale_u);
        check_tile<T>(ws, ws.sa, pw, rs, p, 0);
        pv_tile<T>(lds_v, pw, ws);
    }
}

__device__ __forceinline__ int wave_min(int x)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) x = min(x, __shfl_xor(x, o));
    return x;
}

__device__ __forceinline__ int wave_max(int x)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) x = max(x, __shfl_xor(x, o));
    return x;
}

// Key tiles visited by a workgroup on the general path: the virtual index
// n < len1 maps to tile r1_lo + n, and n >= len1 to tile r2_lo + n - len1.
// A tile t is fully visible for every row when (t + 1) * BN <= pmin or
// lomax <= t * BN and t * BN + BN - 1 <= himin.
struct TileRanges {
    int r1_lo, len1, r2_lo, n;
    int pmin, lomax, himin;
};

// Reduce the rows' visible ranges over the workgroup (wave reductions, then
// one LDS exchange) into the tile ranges. Rows past the end (valid = false)
// do not take part.
template <int BN>
__device__ TileRanges plan_general(RowVis r, bool valid, int (*red)[8], int wave, int lane)
{
    const int big = 0x3fffffff;
    const bool band = valid && r.jlo <= r.jhi;
    int v[6];
    v[0] = valid ? r.pfx : 0;                 // max prefix
    v[1] = valid ? -r.pfx : -big;             // -(min prefix)
    v[2] = band ? -r.jlo : -big;              // -(min band start)
    v[3] = valid ? (band ? r.jlo : big) : -big;  // max band start (empty band: none full)
    v[4] = band ? r.jhi : -big;               // max band end
    v[5] = valid ? (band ? -r.jhi : big) : -big; // -(min band end)
#pragma unroll
    for (int i = 0; i < 6; ++i) v[i] = wave_max(v[i]);
    if (lane == 0) {
#pragma unroll
        for (int i = 0; i < 6; ++i) red[wave][i] = v[i];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 6; ++i)
        v[i] = __builtin_amdgcn_readfirstlane(
            max(max(red[0][i], red[1][i]), max(red[2][i], red[3][i])));
    TileRanges t;
    const int pmax = v[0], lomin = -v[2], himax = v[4];
    t.pmin = -v[1];
    t.lomax = v[3];
    t.himin = -v[5];
    const int a_hi = (pmax + BN - 1) / BN;  // prefix tiles [0, a_hi)
    int b_lo = 0, b_hi = 0;                 // band tiles [b_lo, b_hi)
    if (lomin <= himax) {
        b_lo = lomin / BN;
        b_hi = himax / BN + 1;
    }
    t.r2_lo = 0;
    if (b_lo >= b_hi) {
        t.r1_lo = 0;
        t.len1 = a_hi;
    } else if (a_hi >= b_lo) {  // overlapping or adjacent: one range
        t.r1_lo = a_hi > 0 ? 0 : b_lo;
        t.len1 = max(a_hi, b_hi) - t.r1_lo;
    } else {
        t.r1_lo = 0;
        t.len1 = a_hi;
        t.r2_lo = b_lo;
    }
    t.n = t.len1 + (b_lo < b_hi && a_hi < b_lo ? b_hi - b_lo : 0);
    return t;
}

template <class T>
__global__ __launch_bounds__(NT, 2) void attn_fwd_bf16_kernel(AttnParams p)
{
    constexpr int D = T::D, BN = T::BN;
    // Separate LDS objects per buffer: the compiler can then prove that reads
    // of one buffer do not alias the in-flight direct loads into another.
    __shared__ __attribute__((aligned(1024))) char lds_k0[T::TILE];
    __shared__ __attribute__((aligned(1024))) char lds_k1[T::TILE];
    __shared__ __attribute__((aligned(1024))) char lds_v0[T::TILE];
    __shared__ __attribute__((aligned(1024))) char lds_v1[T::TILE];
    // listed global set: G in LDS, padded with lk to a multiple of BN
    __shared__ __attribute__((aligned(16))) int gl[T::GLIST ? kMaxGlobalList + BN : 4];

    const int tid = threadIdx.x;
    if constexpr (kLdsPoison) {
        const u32x4 ones = {~0u, ~0u, ~0u, ~0u};
        for (int i = tid; i < T::TILE / 16; i += NT) {
            reinterpret_cast<u32x4*>(lds_k0)[i] = ones;
            reinterpret_cast<u32x4*>(lds_k1)[i] = ones;
            reinterpret_cast<u32x4*>(lds_v0)[i] = ones;
            reinterpret_cast<u32x4*>(lds_v1)[i] = ones;
        }
        for (int i = tid; i < (int)(sizeof(gl) / sizeof(int)); i += NT) gl[i] = -1;
        __syncthreads();
    }
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int li = lane & 31, lh = lane >> 5;

    // Read the kernel arguments the set-up needs in one round of scalar loads
    // (the branches below would otherwise spread them over several).
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::"s"(p.compact), "s"(p.map_mode), "s"(p.hp_shift), "s"(p.num_q_tiles), "s"(p.q_order),
                 "s"(p.div_bh.mul), "s"(p.div_bh.shift), "s"(p.div_bh.d), "s"(p.div_hq.mul),
                 "s"(p.div_hq.shift), "s"(p.div_hq.d), "s"(p.div_group.mul),
                 "s"(p.div_group.shift), "s"(p.div_group.d), "s"(p.div_hkv.mul),
                 "s"(p.div_hkv.shift), "s"(p.div_hkv.d), "s"(p.cu_q), "s"(p.seqlen_q),
                 "s"(p.seqlen_k), "s"(p.wg_rows), "s"(p.q), "s"(p.k), "s"(p.v), "s"(p.o),
                 "s"(p.sq_b), "s"(p.sq_h), "s"(p.sq_s), "s"(p.sk_b), "s"(p.sk_h), "s"(p.sk_s),
                 "s"(p.sv_b), "s"(p.sv_h), "s"(p.sv_s), "s"(p.so_h), "s"(p.so_s));
    // Listed global set: the first glob_items workgroups compute the rows
    // whose position is in G (every key visible), wg_rows list entries each,
    // for one head set of one sequence; the others are the ordinary work
    // items, whose rows in G are left to them. Rows that see every key then
    // no longer stretch an ordinary workgroup over the whole key range.
    bool gmode = false;
    WorkItem it;
    if constexpr (T::GLIST) {
        gmode = (int)blockIdx.x < p.glob_items;
        if (gmode) {
            const int e = (int)blockIdx.x;
            const int hsets = p.hq >> p.hp_shift;
            const int c = e % p.glob_chunks, bh = e / p.glob_chunks;
            it.b = bh / hsets;
            it.hq = (bh - it.b * hsets) << p.hp_shift;
            it.hkv = it.hq / p.group;
            it.qt = c;  // chunk of the list
        } else {
            it = decode_block(p, (int)blockIdx.x - p.glob_items);
        }
    } else {
        it = decode_block(p, blockIdx.x);
    }
    int lq, lk;
    int64_t qrow0 = 0, krow0 = 0;  // first token of the sequence (varlen)
    if (p.cu_q) {
        qrow0 = p.cu_q[it.b];
        lq = p.cu_q[it.b + 1] - (int)qrow0;
        krow0 = p.cu_k[it.b];
        lk = p.cu_k[it.b + 1] - (int)krow0;
    } else {
        lq = p.seqlen_q;
        lk = p.seqlen_k;
    }
    const int q0 = gmode ? 0 : it.qt * p.wg_rows;
    if (it.qt < 0 || q0 >= lq) return;  // whole workgroup: no item, or past the sequence's end
    const int hkv = it.hkv;
    // Wave w takes query head hq + (w mod hp) and the 32-row block w / hp of
    // the workgroup's rows (hp = 1: four row blocks of one head; hp = 4: the
    // same 32 rows of four heads that share the K/V tiles).
    const int hq = it.hq + (wave & (p.hp - 1));
    const int rblk = wave >> p.hp_shift;

    const __bf16* qb = static_cast<const __bf16*>(p.q);
    const __bf16* kbase = static_cast<const __bf16*>(p.k);
    const __bf16* vbase = static_cast<const __bf16*>(p.v);
    __bf16* ob = static_cast<__bf16*>(p.o);
    int64_t qoff, koff, voff, ooff;
    if (p.cu_q) {
        qoff = qrow0 * p.sq_s + (int64_t)hq * p.sq_h;
        ooff = qrow0 * p.so_s + (int64_t)hq * p.so_h;
        koff = krow0 * p.sk_s + (int64_t)hkv * p.sk_h;
        voff = krow0 * p.sv_s + (int64_t)hkv * p.sv_h;
    } else {
        qoff = (int64_t)it.b * p.sq_b + (int64_t)hq * p.sq_h;
        ooff = (int64_t)it.b * p.so_b + (int64_t)hq * p.so_h;
        koff = (int64_t)it.b * p.sk_b + (int64_t)hkv * p.sk_h;
        voff = (int64_t)it.b * p.sv_b + (int64_t)hkv * p.sv_h;
    }
    kbase += koff;
    vbase += voff;

    WaveState<T> ws;
    ws.lh = lh;
    // Q fragment: lane holds row q0 + 32*rblk + li (a global row: the row at
    // list entry wg_rows * chunk + 32*rblk + li), dims 16t + 8lh .. +7.
    int qi = q0 + rblk * 32 + li;
    bool row_ok = qi < lq;  // the row exists and this workgroup writes it
    // this sequence's index-mask layout (one shared by all when the stride is 0)
    [[maybe_unused]] const int32_t* gtok = p.gtok ? p.gtok + (int64_t)it.b * p.gtok_stride : nullptr;
    if constexpr (T::GLIST) {
        if (gmode) {
            const int k = it.qt * p.wg_rows + rblk * 32 + li;
            qi = k < p.num_global ? gtok[k] - (lk - lq) : -1;
            row_ok = qi >= 0 && qi < lq;
            if (!row_ok) qi = 0;  // (its Q load stays in range; nothing is written)
        }
    }
    {
        uint32_t bytes = (uint32_t)((((int64_t)lq - 1) * p.sq_s + D) * 2);
        __amdgpu_buffer_rsrc_t qrs = make_rsrc(qb + qoff, bytes);
#pragma unroll
        for (int t = 0; t < T::KSTEPS; ++t) {
            uint32_t off = (uint32_t)(((int64_t)qi * p.sq_s + 16 * t + 8 * lh) * 2);
            ws.qf[t] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(qrs, off, 0, 0));
        }
    }
    // LDS read offsets (within a tile).
    {
        const int r = pi32(li);
#pragma unroll
        for (int t = 0; t < T::KSTEPS; ++t)
            ws.kaddr[t] = r * T::ROWB + (((2 * t + lh) ^ chunk_swizzle<D>(r)) << 4);
        const int g = lane >> 4, sl = lane & 15, a = sl & 3, f = sl >> 2;
        const int sa = ((a & 1) << 1) | (a >> 1);  // head-dim order pi on O^T rows
#pragma unroll
        for (int d = 0; d < T::DBLK; ++d)
#pragma unroll
            for (int rr = 0; rr < 2; ++rr) {
                int key = 8 * (g >> 1) + 4 * rr + f;
                int dd = 32 * d + 16 * (g & 1) + 4 * sa;
                ws.vaddr[d][rr] = key * T::ROWB + (((dd >> 3) ^ chunk_swizzle<D>(key)) << 4) +
                                  (dd & 7) * 2;
            }
    }

    const uint32_t klp = load_lane_offset<T>(wave, lane, p.sk_s);
    const uint32_t vlp = load_lane_offset<T>(wave, lane, p.sv_s);
    // One buffer descriptor per K/V slice; its range ends at the sequence end.
    auto slice_bytes = [&](int64_t stride) {
        return lk <= 0 ? 0u : (uint32_t)((((int64_t)lk - 1) * stride + D) * 2);
    };
    const __amdgpu_buffer_rsrc_t krs = make_rsrc(kbase, slice_bytes(p.sk_s));
    const __amdgpu_buffer_rsrc_t vrs = make_rsrc(vbase, slice_bytes(p.sv_s));
    const uint32_t krow = (uint32_t)(p.sk_s * 2), vrow = (uint32_t)(p.sv_s * 2);

    // Visible keys of this lane's row; rows past the end see nothing.
    ws.ip = qi + (lk - lq);
    ws.pfx = 0;
    ws.jlo = 1;
    ws.jhi = 0;
    TileRanges tr = {};
    int jbeg, jend;
    TilePlan gp = {};
    int ng = 0;
    if constexpr (T::GEN) {
        __shared__ int red[4][8];
        const int32_t* seg = p.seg ? p.seg + (int64_t)it.b * p.seg_stride : nullptr;
        if (seg) {  // stage the segment starts in the (not yet used) V buffer 1
            int32_t* sl = reinterpret_cast<int32_t*>(lds_v1);
            for (int i = tid; i < p.num_seg; i += NT) sl[i] = seg[i];
            __syncthreads();
            seg = sl;
        }
        if constexpr (T::GLIST) {
            ng = p.num_global;
            const int npad = (ng + BN - 1) / BN * BN;
            for (int i = tid; i < npad; i += NT) gl[i] = i < ng ? gtok[i] : lk;
            __syncthreads();
        }
        RowVis rv = {0, 1, 0};
        if (row_ok) {
            if constexpr (T::GLIST) {
                if (gmode) {
                    rv.jlo = 0;
                    rv.jhi = lk - 1;
                } else if (listed(gl, ng, qi + (lk - lq))) {
                    row_ok = false;  // a row of G: the global-row items write it
                } else {
                    rv = row_vis_listed(p.band, gl, ng, qi, lq, lk);
                }
            } else
                rv = row_visibility(p.mask_kind, p.band, p.num_global, seg, p.num_seg,
                                    p.query_start, qi, lq, lk);
        }
        ws.pfx = rv.pfx;
        ws.jlo = rv.jlo;
        ws.jhi = rv.jhi;
        tr = plan_general<BN>(rv, row_ok, red, wave, lane);
        jbeg = 0;
        jend = tr.n;
    } else {
        if (qi < lq) band_row(p.band, qi, lq, lk, &ws.jlo, &ws.jhi);
        gp = plan_tiles(p.band, q0, p.wg_rows, lq, lk, BN);
        jbeg = gp.lo;
        jend = gp.hi;
    }
    // DIAG: visited tiles, as virtual indices n = 0 .. hi - lo - 1, run from
    // the tile of the workgroup's last row down to lo, then from there up
    // (tile_of below); a tile is left of every row when its last key is at or
    // before the first row's key-axis position, right when its first key is
    // at or after the last row's.
    int t_diag = 0, n_desc = 0, ip_first = 0, ip_last = 0;
    if constexpr (T::DIAG) {
        ip_first = q0 + (lk - lq);
        ip_last = min(q0 + p.wg_rows, lq) - 1 + (lk - lq);
        t_diag = min(max(ip_last, 0) / BN, gp.hi - 1);
        if (t_diag < gp.lo) t_diag = gp.lo;
        n_desc = t_diag - gp.lo + 1;
        jbeg = 0;
        jend = gp.hi - gp.lo;
    }
    // Relative-position reference: the row's first visible key for softmax
    // (largest bias; the shift is added back to the LSE), i' otherwise.
    ws.jref = T::SOFTMAX ? (ws.pfx > 0 ? 0 : ws.jlo) : ws.ip;
    if constexpr (T::GLIST && T::SOFTMAX) {  // the smallest visible key may be one of G
        int jr = ws.jlo <= ws.jhi ? ws.jlo : 0x7fffffff;
        if (ng > 0 && gl[0] < lk) jr = min(jr, gl[0]);
        ws.jref = jr == 0x7fffffff ? 0 : jr;
    }
    ws.bias_abs = 0.0f;
    ws.bias_lin = 0.0f;
    if constexpr (T::BIAS == kBiasAlibi) ws.bias_abs = -p.slopes[hq] * p.unit;
    if constexpr (T::BIAS == kBiasRelPos) ws.bias_lin = p.unit;
    if constexpr (T::BIAS == kBiasGeneral) {
        if (p.slopes) ws.bias_abs = -p.slopes[hq] * p.unit;
        if (p.relpos) ws.bias_lin = p.unit;
    }

#pragma unroll
    for (int d = 0; d < T::DBLK; ++d) ws.oacc[d] = f32x16{};
    ws.m_run = -__builtin_inff();
    ws.l_run = 0.0f;
    ws.l_o = 0.0f;
    ws.alpha = 1.0f;
    ws.need = false;

    // Key tile of loop index n, and (general path) whether it is fully visible.
    auto tile_of = [&](int n) __attribute__((always_inline)) -> int {
        if constexpr (T::GEN)
            return n < tr.len1 ? tr.r1_lo + n : tr.r2_lo + (n - tr.len1);
        else if constexpr (T::DIAG)
            return n < n_desc ? t_diag - n : gp.lo + n;
        else
            return n;
    };
    // DIAG: class of a tile: masked (any side), or check-free on the given side
    auto diag_class = [&](int t) __attribute__((always_inline)) -> int {
        if (!(t >= gp.full_lo && t < gp.full_hi)) return 0;
        if ((t + 1) * BN - 1 <= ip_first) return 1 + kSideLeft;
        if (t * BN >= ip_last) return 1 + kSideRight;
        return 1 + kSideBoth;
    };
    auto gen_full = [&](int t) __attribute__((always_inline)) -> bool {
        return (t + 1) * BN <= tr.pmin || (tr.lomax <= t * BN && t * BN + BN - 1 <= tr.himin);
    };

    if (jend > jbeg) {
        // Prologue: K_lo, V_lo -> buffers 0, K_lo+1 -> K buffer 1; S_lo.
        const int t0 = tile_of(jbeg);
        issue_tile<T>(lds_k0, krs, t0 * BN, krow, klp, wave);
        issue_tile<T>(lds_v0, vrs, t0 * BN, vrow, vlp, wave);
        // past the last tile K_lo+1 reads rows beyond the sequence end (zeros)
        issue_tile<T>(lds_k1, krs, jbeg + 1 < jend ? tile_of(jbeg + 1) * BN : lk, krow, klp, wave);
        // Q and K_lo have landed (V_lo and K_lo+1, the last 2 LOADS direct
        // loads, may still be in flight: the barrier after the first tile's
        // max waits for them)
        __builtin_amdgcn_s_waitcnt(vmcnt_only(2 * T::LOADS));
        asm volatile("s_barrier" ::: "memory");  // no LDS access moves across it
        qk_tile<T>(lds_k0, ws, ws.sa);
        bool masked_lo;
        if constexpr (T::GEN)
            masked_lo = !gen_full(t0);
        else
            masked_lo = !(t0 >= gp.full_lo && t0 < gp.full_hi);
        // the running max starts at the first tile's max (-inf for rows that
        // see none of its keys)
        const float mx = masked_lo ? mods_and_max<T, true>(ws.sa, p, ws, t0 * BN)
                                   : mods_and_max<T, false>(ws.sa, p, ws, t0 * BN);
        if constexpr (T::MAXFREE)
            ws.m_run = mx;
        else
            update_max(ws, mx);
        if constexpr (T::FOLD) {  // take the running max off the first tile's scores
            const float mb = mx == -__builtin_inff() ? 0.0f : mx;
#pragma unroll
            for (int b = 0; b < T::NB; ++b)
#pragma unroll
                for (int e = 0; e < 16; ++e) ws.sa[b][e] -= mb;
        }
        __syncthreads();  // K buffer 0 is reloaded in the first iteration

        // Iteration j with parity PAR = (j - jbeg) & 1 reads K_{j+1} from K
        // buffer PAR^1 and V_j from V buffer PAR, and loads K_{j+2} into K
        // buffer PAR and V_{j+1} into V buffer PAR^1 (j counts visited
        // tiles). MASKED is the class of tile j+1.
        auto iteration = [&](auto par_c, auto masked_c, auto side_c, int j)
                             __attribute__((always_inline)) {
            constexpr int PAR = decltype(par_c)::value;
            constexpr bool MASKED = decltype(masked_c)::value;
            constexpr int SIDE = decltype(side_c)::value;
            char* kread = PAR ? lds_k0 : lds_k1;
            char* kwrite = PAR ? lds_k1 : lds_k0;
            char* vread = PAR ? lds_v1 : lds_v0;
            char* vwrite = PAR ? lds_v0 : lds_v1;
            rescale_if_needed(ws);
            const int t1 = tile_of(j + 1);
            // past the last tile the K load reads rows beyond the sequence end (zeros)
            const int jk = j + 2 < jend ? tile_of(j + 2) * BN : lk;
            auto load = [&](int i) __attribute__((always_inline)) {
                if (i < T::LOADS)
                    issue_load<T>(kwrite, krs, jk, krow, klp, wave, i);
                else
                    issue_load<T>(vwrite, vrs, t1 * BN, vrow, vlp, wave, i - T::LOADS);
            };
            const float m_use = ws.m_run == -__builtin_inff() ? 0.0f : ws.m_run;
            if constexpr (PAR == 0)
                pipelined_step<T, MASKED, SIDE>(kread, vread, ws, ws.sa, ws.sb, p, m_use,
                                                tile_of(j) * BN, t1 * BN, load);
            else
                pipelined_step<T, MASKED, SIDE>(kread, vread, ws, ws.sb, ws.sa, p, m_use,
                                                tile_of(j) * BN, t1 * BN, load);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
        };
        // Loop splitting (Section 3.4): runs of partial and check-free tiles,
        // each phase with a branch-free body.
        int j = jbeg, par = 0;
        // iterations while tile j+1 < end, with the side of those tiles
        auto phase = [&](auto masked_c, int end, auto side_c) __attribute__((always_inline)) {
            if (par && j + 1 < end) {
                iteration(Parity<1>{}, masked_c, side_c, j);
                ++j;
                par = 0;
            }
            while (j + 2 < end) {
                iteration(Parity<0>{}, masked_c, side_c, j);
                iteration(Parity<1>{}, masked_c, side_c, j + 1);
                j += 2;
            }
            if (j + 1 < end) {
                iteration(Parity<0>{}, masked_c, side_c, j);
                ++j;
                par = 1;
            }
        };
        using Both = std::integral_constant<int, kSideBoth>;
        if constexpr (T::GEN) {
            // Visited tiles fall into at most four runs: check-free prefix
            // tiles, partial tiles, check-free band tiles, partial tiles. Any
            // further check-free tile goes through the masked body, which is
            // correct for every tile.
            auto run_end = [&](int from, bool full) __attribute__((always_inline)) {
                int e = from;
                while (e < jend && gen_full(tile_of(e)) == full) ++e;
                return e;
            };
            const int e1 = run_end(jbeg + 1, true);
            const int e2 = run_end(e1, false);
            const int e3 = run_end(e2, true);
            phase(Bool<false>{}, e1, Both{});
            phase(Bool<true>{}, e2, Both{});
            phase(Bool<false>{}, e3, Both{});
            phase(Bool<true>{}, jend, Both{});
        } else if constexpr (T::DIAG) {
            // In visiting order: tiles around the diagonal (partial or
            // check-free on neither side), check-free tiles left of every row,
            // partial ones at the low end, check-free tiles right of every
            // row, partial ones at the high end. Each phase takes the run of
            // its class that starts at the next tile; the masked body, which
            // is correct for every tile, finishes whatever remains.
            auto run_end = [&](int from, int cls) __attribute__((always_inline)) {
                int e = from;
                while (e < jend && diag_class(tile_of(e)) == cls) ++e;
                return e;
            };
            using Left = std::integral_constant<int, kSideLeft>;
            using Right = std::integral_constant<int, kSideRight>;
            phase(Bool<true>{}, run_end(j + 1, 0), Both{});
            phase(Bool<false>{}, run_end(j + 1, 1 + kSideBoth), Both{});
            phase(Bool<true>{}, run_end(j + 1, 0), Both{});
            phase(Bool<false>{}, run_end(j + 1, 1 + kSideLeft), Left{});
            phase(Bool<true>{}, run_end(j + 1, 0), Both{});
            phase(Bool<false>{}, run_end(j + 1, 1 + kSideRight), Right{});
            phase(Bool<true>{}, jend, Both{});
        } else {
            phase(Bool<true>{}, gp.full_lo, Both{});
            phase(Bool<false>{}, gp.full_hi, Both{});
            phase(Bool<true>{}, jend, Both{});
        }
        rescale_if_needed(ws);
        const float m_use = ws.m_run == -__builtin_inff() ? 0.0f : ws.m_run;
        if (par)
            last_step<T>(lds_v1, ws, ws.sb, p, m_use, tile_of(j) * BN);
        else
            last_step<T>(lds_v0, ws, ws.sa, p, m_use, tile_of(j) * BN);
    }
    if constexpr (T::GLIST)
        if (!gmode)  // (global rows see every key through the planned tiles)
            gathered_tiles<T>(ws, p, gl, ng, lds_k0, lds_v0, krs, vrs, krow, vrow, lk, row_ok, wave,
                          lane);

    // Epilogue. Softmax: O = O^T / l (with PSUM_BF16 the sum of the bf16 P
    // O was made from), LSE = (m + log2 l) ln 2 with the fp32 l (+ the relative
    // position shift); lane halves hold halves of the row sums. ReLU /
    // Sigmoid: O = O^T / L.
    float inv = 0.0f;
    float l_tot = 0.0f;
    if constexpr (T::SOFTMAX) {
        l_tot = pair_sum(ws.l_run);
        const float lo_tot = T::PSUM_BF16 ? pair_sum(ws.l_o) : l_tot;
        inv = l_tot > 0.0f && lo_tot > 0.0f ? 1.0f / lo_tot : 0.0f;
    } else {
        inv = lk > 0 ? 1.0f / (float)lk : 0.0f;
    }
    if (row_ok) {
        __bf16* orow = ob + ooff + (int64_t)qi * p.so_s;
#pragma unroll
        for (int d = 0; d < T::DBLK; ++d) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                u32x4 w;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w[q] = pack_bf16(ws.oacc[d][8 * u + 2 * q] * inv, ws.oacc[d][8 * u + 2 * q + 1] * inv);
                *reinterpret_cast<u32x4*>(orow + 32 * d + 16 * u + 8 * lh) = w;
            }
        }
        if constexpr (T::SOFTMAX) {
            if (p.lse && lh == 0) {
                float lse = -__builtin_inff();
                if (l_tot > 0.0f) {
                    lse = (ws.m_run + __builtin_log2f(l_tot)) * kLn2;
                    if (ws.bias_lin != 0.0f) lse += (float)(ws.ip - ws.jref);
                }
                int64_t idx = p.cu_q ? (int64_t)hq * p.total_q + qrow0 + qi
                                     : ((int64_t)it.b * p.hq + hq) * lq + qi;
                p.lse[idx] = lse;
            }
        }
    }
}

// Keys per tile. 64 halves the per-tile barrier, load-wait and max-exchange
// overhead relative to 32 and still fits the pipeline's double-buffered
// scores in the registers of two waves per SIMD.
constexpr int key_tile_width(int) { return 64; }

template <int D, int CAP, int BIAS, int NORM, bool GEN, bool LEFT = true, bool GLIST = false>
hipError_t launch_variant(const AttnParams& p, hipStream_t stream)
{
    using T = Traits<D, key_tile_width(D), CAP, BIAS, NORM, GEN, LEFT, GLIST>;
    hipLaunchKernelGGL((attn_fwd_bf16_kernel<T>), dim3((unsigned)p.grid), dim3(NT), 0, stream, p);
    return hipGetLastError();
}

// Calls f(std::integral_constant<int, kCap*>) for the soft-cap form of the
// launch: off, the short form up to C = kCapShortMax, the exact one above.
template <class F>
hipError_t with_cap(const AttnParams& p, F&& f)
{
    if (p.softcap <= 0.0f) return f(std::integral_constant<int, kCapOff>{});
    // (the short form's kernels that fold the running max take the soft-cap
    // from a polynomial whose coefficients must be normal floats)
    if (p.softcap <= kCapShortMax && p.cap_zmax >= 0.0f)
        return f(std::integral_constant<int, kCapShort>{});
    return f(std::integral_constant<int, kCapExact>{});
}

// The general-path instantiations of one normalisation: head dim, soft-cap,
// and a runtime-coefficient bias when ALiBi or the relative position is on;
// GLIST for a listed global set.
template <int NORM, bool GLIST = false>
hipError_t launch_general_norm(const AttnParams& p, int head_dim, hipStream_t stream)
{
    const bool bias = p.slopes != nullptr || p.relpos != 0;
    return with_cap(p, [&](auto cap) {
        constexpr int C = decltype(cap)::value;
        if (head_dim == 128)
            return bias ? launch_variant<128, C, kBiasGeneral, NORM, true, true, GLIST>(p, stream)
                        : launch_variant<128, C, kBiasNone, NORM, true, true, GLIST>(p, stream);
        return bias ? launch_variant<64, C, kBiasGeneral, NORM, true, true, GLIST>(p, stream)
                    : launch_variant<64, C, kBiasNone, NORM, true, true, GLIST>(p, stream);
    });
}

}  // namespace
}  // namespace attn

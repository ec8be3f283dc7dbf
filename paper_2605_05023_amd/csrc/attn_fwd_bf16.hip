// attn_fwd_bf16.hip -- fused attention forward for bf16 inputs on gfx950.
//
// One workgroup computes BM = 128 query rows of one (sequence, query head):
// four wavefronts of 32 rows each. It streams the key/value tiles of BN = 64
// keys that the mask leaves visible through LDS (double-buffered), computes
// the tile's scores on the bf16 matrix cores with fp32 accumulation, applies
// the score modifications and, on partial tiles only, the mask in registers,
// keeps an online softmax per row, and accumulates P V on the matrix cores
// (Eq. 1 and 2 of Section 2.2; the Score / Mask / Norm stages of Appendix A;
// loop splitting of Section 3.4 and block skipping of Appendix C).
//
// Layout choices for the 64-wide wavefront and v_mfma_f32_32x32x16_bf16:
//  * Scores are computed transposed, S^T = K Q^T, so a lane owns one query
//    row (lane % 32) and 16 keys per 32-key block. The row max and row sum
//    are then per-lane reductions plus one exchange with lane ^ 32.
//  * K rows are fed to the A operand in the order pi(r) (bits 2 and 3 of the
//    row index swapped). With that order the accumulator of lane half h holds
//    keys 8h..8h+7 and 16+8h..16+8h+7 of the block in registers 0..7 and 8..15,
//    which is exactly the B-operand layout of the P V product. P never leaves
//    the registers.
//  * V is stored transposed in LDS (V^T, keys contiguous) so the A operand of
//    O^T = V^T P^T is one 16-byte LDS read per lane; the transpose happens in
//    registers while the tile is staged from global memory.
//  * O^T rows (head-dim) go through the same pi order, so a lane ends with 8
//    consecutive head-dim values per half block: 16-byte stores.
//  * LDS rows use an XOR swizzle of their 16-byte chunks so the A-operand
//    reads of 8 consecutive lanes hit 8 distinct bank groups.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernel_params.h"
#include "launch.h"
#include "score_mods.h"

namespace attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = 128;    // query rows per workgroup
constexpr int BN = 64;     // keys per tile
constexpr int NT = 256;    // threads per workgroup (4 waves)
constexpr float TAU = 8.0f;  // lazy-rescale threshold, log2 units

// pi: swap bits 2 and 3 of a row index within a 32-row block.
__device__ __forceinline__ int pi32(int r)
{
    return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes)
{
    // dword3 0x00020000: 32-bit untyped data format, no swizzle (gfx9 family)
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             0x00020000);
}

template <int D>
struct Cfg {
    static constexpr int CHUNKS = D / 8;                 // 16-byte chunks per K row
    static constexpr int K_BYTES = BN * D * 2;           // one K tile
    static constexpr int V_BYTES = D * BN * 2;           // one V^T tile
    static constexpr int STAGE = K_BYTES + V_BYTES;
    static constexpr int K_PASSES = BN * CHUNKS / NT;    // 16-byte K loads per thread
    static constexpr int V_KPT = BN * D / (8 * NT);      // keys per thread in the V transpose
    static constexpr int V_GROUPS = BN / V_KPT;          // key groups per d-chunk
    static constexpr int KSTEPS = D / 16;                // MFMA k-steps over the head dim
    static constexpr int DBLK = D / 32;                  // 32-row blocks of O^T
    static_assert(K_PASSES * NT == BN * CHUNKS, "K tile split");
    static_assert(V_GROUPS * (D / 8) == NT, "V tile split");
};

// Byte offset of chunk c of K row r inside a K tile.
template <int D>
__device__ __forceinline__ int k_off(int r, int c)
{
    constexpr int mask = (D / 8) - 1;
    return r * D * 2 + ((c ^ (pi32(r & 31) & mask)) << 4);
}

// Byte offset of key byte `kb` (0..127) of V^T row d inside a V^T tile.
__device__ __forceinline__ int vt_off(int d, int kbyte)
{
    int c = kbyte >> 4;
    return d * (BN * 2) + (((c ^ (pi32(d & 31) & 7)) << 4) | (kbyte & 15));
}

template <int D>
struct TileRegs {
    u32x4 k[Cfg<D>::K_PASSES];
    u32x4 v[Cfg<D>::V_KPT];
};

// Issue the global loads of key tile `kt` (rows j0..j0+BN-1) into registers.
// Rows at or past the sequence end fall outside the buffer range and read 0.
template <int D>
__device__ __forceinline__ void load_tile(TileRegs<D>& r, __amdgpu_buffer_rsrc_t krs,
                                          __amdgpu_buffer_rsrc_t vrs, int j0, int64_t ks,
                                          int64_t vs, int tid)
{
    using C = Cfg<D>;
#pragma unroll
    for (int p = 0; p < C::K_PASSES; ++p) {
        int ci = p * NT + tid;
        int row = ci / C::CHUNKS, ch = ci % C::CHUNKS;
        uint32_t off = (uint32_t)(((int64_t)(j0 + row) * ks + ch * 8) * 2);
        r.k[p] = __builtin_amdgcn_raw_buffer_load_b128(krs, off, 0, 0);
    }
    int kg = tid % C::V_GROUPS, dc = tid / C::V_GROUPS;
#pragma unroll
    for (int u = 0; u < C::V_KPT; ++u) {
        int row = kg * C::V_KPT + u;
        uint32_t off = (uint32_t)(((int64_t)(j0 + row) * vs + dc * 8) * 2);
        r.v[u] = __builtin_amdgcn_raw_buffer_load_b128(vrs, off, 0, 0);
    }
}

// Write staged registers into one LDS stage: K as rows, V transposed.
template <int D>
__device__ __forceinline__ void store_tile(const TileRegs<D>& r, char* stage, int tid)
{
    using C = Cfg<D>;
#pragma unroll
    for (int p = 0; p < C::K_PASSES; ++p) {
        int ci = p * NT + tid;
        int row = ci / C::CHUNKS, ch = ci % C::CHUNKS;
        *reinterpret_cast<u32x4*>(stage + k_off<D>(row, ch)) = r.k[p];
    }
    char* vt = stage + C::K_BYTES;
    int kg = tid % C::V_GROUPS, dc = tid / C::V_GROUPS;
    int kbyte = kg * C::V_KPT * 2;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            int d = dc * 8 + 2 * m + e;
            if constexpr (C::V_KPT == 4) {
                u32x2 w;
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    uint32_t a = r.v[2 * q][m], b = r.v[2 * q + 1][m];
                    w[q] = e == 0 ? ((a & 0xffffu) | (b << 16)) : ((a >> 16) | (b & 0xffff0000u));
                }
                *reinterpret_cast<u32x2*>(vt + vt_off(d, kbyte)) = w;
            } else {
                static_assert(C::V_KPT == 2, "V transpose width");
                uint32_t a = r.v[0][m], b = r.v[1][m];
                uint32_t w = e == 0 ? ((a & 0xffffu) | (b << 16)) : ((a >> 16) | (b & 0xffff0000u));
                *reinterpret_cast<uint32_t*>(vt + vt_off(d, kbyte)) = w;
            }
        }
    }
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b)
{
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 v;
    v[0] = (__bf16)a;
    v[1] = (__bf16)b;
    return __builtin_bit_cast(uint32_t, v);
}

struct WorkItem {
    int b, hq, qt;
};

// Map the hardware workgroup id to (sequence, query head, query tile).
// Query tiles are issued longest-first (the last tiles of a causal sequence
// see the most keys). Mode 1 keeps all query heads of a kv-head group on one
// XCD (workgroup ids are dealt round-robin over the 8 XCDs), so their K/V
// tiles are shared through that XCD's L2.
__device__ __forceinline__ WorkItem decode_block(const AttnParams& p, int w)
{
    WorkItem it;
    int nbh = p.batch * p.hq;
    if (p.map_mode == 1) {
        int x = w & 7, k = w >> 3;
        int groups_per_xcd = (p.batch * p.hkv) >> 3;
        int per_tile = groups_per_xcd * p.group;
        int qt_rev = k / per_tile, rem = k % per_tile;
        int gi = rem / p.group, r = rem % p.group;
        int g = x + 8 * gi;
        it.b = g / p.hkv;
        it.hq = (g % p.hkv) * p.group + r;
        it.qt = p.num_q_tiles - 1 - qt_rev;
    } else {
        int qt_rev = w / nbh, rem = w % nbh;
        it.b = rem / p.hq;
        it.hq = rem % p.hq;
        it.qt = p.num_q_tiles - 1 - qt_rev;
    }
    return it;
}

// One key tile for one wavefront: S^T = K Q^T on the matrix cores, score
// mods, the element mask when MASKED (partial tiles only), online softmax with
// lazy rescaling, then O^T += V^T P^T.
template <int D, bool SOFTCAP, bool ALIBI, bool MASKED>
__device__ __forceinline__ void tile_step(const char* st, const bf16x8 (&qf)[Cfg<D>::KSTEPS],
                                          f32x16 (&oacc)[Cfg<D>::DBLK], float& m_run, float& l_run,
                                          const AttnParams& p, int j0, int li, int lh, int jlo,
                                          int jhi, int ip, float slope_log2)
{
    using C = Cfg<D>;
    f32x16 sacc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[b][e] = 0.0f;
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            int r = 32 * b + pi32(li);
            bf16x8 a = *reinterpret_cast<const bf16x8*>(st + k_off<D>(r, 2 * t + lh));
            sacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[t], sacc[b], 0, 0, 0);
        }
    }
    // Element (b, e) is key j0 + 32b + 8lh + e + (e >= 8 ? 8 : 0).
    constexpr bool MODS = SOFTCAP || ALIBI;
    float mx = -__builtin_inff();
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            int j = j0 + 32 * b + 8 * lh + e + (e >= 8 ? 8 : 0);
            float x = sacc[b][e];
            if constexpr (MODS)
                x = score_log2<SOFTCAP, ALIBI>(x, p.scale_log2, p.softcap_pre, p.softcap_post,
                                               slope_log2, ip, j);
            if constexpr (MASKED)
                if (j < jlo || j > jhi) x = -__builtin_inff();
            sacc[b][e] = x;
            mx = __builtin_fmaxf(mx, x);
        }
    }
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 32));
    if constexpr (!MODS) mx *= p.scale_log2;  // raw max -> log2 units (scale > 0)
    const float m_new = __builtin_fmaxf(m_run, mx);
    const bool need = m_new > m_run + TAU;
    if (__builtin_amdgcn_ballot_w64(need)) {
        float alpha = need ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
        if (need) m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < C::DBLK; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) oacc[d][e] *= alpha;
    }
    const float m_use = m_run == -__builtin_inff() ? 0.0f : m_run;
    float rs = 0.0f;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            float x = sacc[b][e];
            float y = MODS ? x - m_use : __builtin_fmaf(x, p.scale_log2, -m_use);
            float pe = __builtin_amdgcn_exp2f(y);
            sacc[b][e] = pe;
            rs += pe;
        }
    }
    l_run += rs;
    // O^T += V^T P^T over four 16-key steps.
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            u32x4 pw;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                pw[q] = pack_bf16(sacc[b][8 * u + 2 * q], sacc[b][8 * u + 2 * q + 1]);
            bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
            int kbyte = (32 * b + 16 * u + 8 * lh) * 2;
#pragma unroll
            for (int d = 0; d < C::DBLK; ++d) {
                int dr = 32 * d + pi32(li);
                bf16x8 a = *reinterpret_cast<const bf16x8*>(st + C::K_BYTES + vt_off(dr, kbyte));
                oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, oacc[d], 0, 0, 0);
            }
        }
    }
}

template <int D, bool SOFTCAP, bool ALIBI>
__global__ __launch_bounds__(NT, 2) void attn_fwd_bf16_kernel(AttnParams p)
{
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) char smem[2 * C::STAGE];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int li = lane & 31, lh = lane >> 5;

    const WorkItem it = decode_block(p, blockIdx.x);
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
    const int q0 = it.qt * BM;
    if (q0 >= lq) return;  // whole workgroup: tile past this sequence's end
    const int hkv = it.hq / p.group;

    const __bf16* qb = static_cast<const __bf16*>(p.q);
    const __bf16* kb = static_cast<const __bf16*>(p.k);
    const __bf16* vb = static_cast<const __bf16*>(p.v);
    __bf16* ob = static_cast<__bf16*>(p.o);
    int64_t qoff, koff, voff, ooff;
    if (p.cu_q) {
        qoff = qrow0 * p.sq_s + (int64_t)it.hq * p.sq_h;
        ooff = qrow0 * p.so_s + (int64_t)it.hq * p.so_h;
        koff = krow0 * p.sk_s + (int64_t)hkv * p.sk_h;
        voff = krow0 * p.sv_s + (int64_t)hkv * p.sv_h;
    } else {
        qoff = (int64_t)it.b * p.sq_b + (int64_t)it.hq * p.sq_h;
        ooff = (int64_t)it.b * p.so_b + (int64_t)it.hq * p.so_h;
        koff = (int64_t)it.b * p.sk_b + (int64_t)hkv * p.sk_h;
        voff = (int64_t)it.b * p.sv_b + (int64_t)hkv * p.sv_h;
    }
    // Buffer ranges cover exactly the rows of this sequence and head.
    auto rows_bytes = [](int rows, int64_t stride) -> uint32_t {
        return rows <= 0 ? 0u : (uint32_t)((((int64_t)rows - 1) * stride + D) * 2);
    };
    const __amdgpu_buffer_rsrc_t qrs = make_rsrc(qb + qoff, rows_bytes(lq, p.sq_s));
    const __amdgpu_buffer_rsrc_t krs = make_rsrc(kb + koff, rows_bytes(lk, p.sk_s));
    const __amdgpu_buffer_rsrc_t vrs = make_rsrc(vb + voff, rows_bytes(lk, p.sv_s));

    // Q fragment (B operand): lane holds row q0 + 32*wave + li, dims 16t + 8lh .. +7.
    const int qi = q0 + wave * 32 + li;
    bf16x8 qf[C::KSTEPS];
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) {
        uint32_t off = (uint32_t)(((int64_t)qi * p.sq_s + 16 * t + 8 * lh) * 2);
        u32x4 raw = __builtin_amdgcn_raw_buffer_load_b128(qrs, off, 0, 0);
        qf[t] = __builtin_bit_cast(bf16x8, raw);
    }

    // Visible key interval of this lane's row; rows past the end see nothing.
    int jlo = 1, jhi = 0;
    if (qi < lq) band_row(p.band, qi, lq, lk, &jlo, &jhi);
    const int ip = qi + (lk - lq);
    float slope_log2 = 0.0f;
    if constexpr (ALIBI) slope_log2 = p.slopes[it.hq] * kLog2e;

    const TilePlan gp = plan_tiles(p.band, q0, BM, lq, lk, BN);
    const TilePlan wp = plan_tiles(p.band, q0 + wave * 32, 32, lq, lk, BN);

    f32x16 oacc[C::DBLK];
#pragma unroll
    for (int d = 0; d < C::DBLK; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[d][e] = 0.0f;
    float m_run = -__builtin_inff();
    float l_run = 0.0f;

    if (gp.hi > gp.lo) {
        TileRegs<D> regs;
        load_tile<D>(regs, krs, vrs, gp.lo * BN, p.sk_s, p.sv_s, tid);
        store_tile<D>(regs, smem, tid);
        __syncthreads();
        int stage = 0;
        for (int kt = gp.lo; kt < gp.hi; ++kt) {
            const bool has_next = kt + 1 < gp.hi;
            if (has_next) load_tile<D>(regs, krs, vrs, (kt + 1) * BN, p.sk_s, p.sv_s, tid);
            const char* st = smem + stage * C::STAGE;
            const bool active = kt >= wp.lo && kt < wp.hi;
            if (active) {
                const bool masked = !(kt >= wp.full_lo && kt < wp.full_hi);
                if (masked)
                    tile_step<D, SOFTCAP, ALIBI, true>(st, qf, oacc, m_run, l_run, p, kt * BN, li, lh,
                                                       jlo, jhi, ip, slope_log2);
                else
                    tile_step<D, SOFTCAP, ALIBI, false>(st, qf, oacc, m_run, l_run, p, kt * BN, li, lh,
                                                        jlo, jhi, ip, slope_log2);
            }
            if (has_next) store_tile<D>(regs, smem + (stage ^ 1) * C::STAGE, tid);
            __syncthreads();
            stage ^= 1;
        }
    }

    // Epilogue: O = O^T / l, LSE = (m + log2 l) ln 2. Lane halves hold halves of the row sum.
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (qi < lq) {
        const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
        __bf16* orow = ob + ooff + (int64_t)qi * p.so_s;
#pragma unroll
        for (int d = 0; d < C::DBLK; ++d) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                u32x4 w;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w[q] = pack_bf16(oacc[d][8 * u + 2 * q] * inv, oacc[d][8 * u + 2 * q + 1] * inv);
                *reinterpret_cast<u32x4*>(orow + 32 * d + 16 * u + 8 * lh) = w;
            }
        }
        if (p.lse && lh == 0) {
            float lse = l_tot > 0.0f ? (m_run + __builtin_log2f(l_tot)) * kLn2 : -__builtin_inff();
            int64_t idx = p.cu_q ? (int64_t)it.hq * p.total_q + qrow0 + qi
                                 : ((int64_t)it.b * p.hq + it.hq) * lq + qi;
            p.lse[idx] = lse;
        }
    }
}

template <int D, bool SOFTCAP, bool ALIBI>
hipError_t launch(const AttnParams& p, hipStream_t stream)
{
    int64_t blocks = (int64_t)p.num_q_tiles * p.hq * p.batch;
    hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, SOFTCAP, ALIBI>), dim3((unsigned)blocks), dim3(NT),
                       0, stream, p);
    return hipGetLastError();
}

}  // namespace

int bf16_block_m() { return BM; }

hipError_t launch_bf16(const AttnParams& p, int head_dim, hipStream_t stream)
{
    const bool sc = p.softcap > 0.0f, al = p.slopes != nullptr;
    if (head_dim == 128) {
        if (sc && al) return launch<128, true, true>(p, stream);
        if (sc) return launch<128, true, false>(p, stream);
        if (al) return launch<128, false, true>(p, stream);
        return launch<128, false, false>(p, stream);
    }
    if (sc && al) return launch<64, true, true>(p, stream);
    if (sc) return launch<64, true, false>(p, stream);
    if (al) return launch<64, false, true>(p, stream);
    return launch<64, false, false>(p, stream);
}

}  // namespace attn

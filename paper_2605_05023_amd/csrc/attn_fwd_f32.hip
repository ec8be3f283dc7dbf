// attn_fwd_f32.hip -- fused attention forward for fp32 inputs on gfx950.
//
// fp32 has no faster matrix path on this chip (the fp32 matrix and vector
// peaks are equal), so each lane owns one query row and accumulates with
// fp32 vector FMAs. A workgroup covers 64 query rows of one (sequence, query
// head) with four wavefronts that split the key tiles between them (wave w
// takes tiles lo + w, lo + w + 4, ...), each staging its own key/value tiles
// through LDS and reading them as broadcasts; the four partial results
// (running max, sum and O per row) are merged through LDS at the end. The score modifications, the masks with
// tile skipping, the base-2 online softmax and the ReLU / Sigmoid
// normalisations are the same as in the bf16 kernel (Eq. 1 and 2 of Section
// 2.2, Appendix A). On the general mask path each lane derives its row's
// visible keys (row_vis.h) and the wave visits the union of the rows' tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernel_params.h"
#include "launch.h"
#include "row_vis.h"
#include "score_mods.h"

namespace attn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 64;     // query rows per workgroup (one per lane of every wave)
constexpr int NW = 4;      // wavefronts, each with a share of the key tiles
constexpr int NT = 64 * NW;

// Keys per tile: the four waves' double K/V tiles fit 64 KiB of LDS.
constexpr int key_tile(int d) { return d == 128 ? 16 : 32; }

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

template <int D, bool SOFTCAP, int BIAS, int NORM, bool GEN>
__global__ __launch_bounds__(NT) void attn_fwd_f32_kernel(AttnParams p)
{
    constexpr bool SOFTMAX = NORM == kNormSoftmax;
    constexpr int BN = key_tile(D);
    constexpr int KV_BYTES = NW * 2 * BN * D * 4;         // per-wave K and V tiles
    constexpr int MERGE_BYTES = 2 * BM * (D + 2) * 4;      // two partial results
    __shared__ __attribute__((aligned(16))) float qs[BM][D + 4];  // padded rows
    __shared__ __attribute__((aligned(16))) char lds[KV_BYTES > MERGE_BYTES ? KV_BYTES : MERGE_BYTES];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    if constexpr (kLdsPoison) {
        for (int i = tid; i < (int)(sizeof(qs) / 4); i += NT) (&qs[0][0])[i] = __builtin_bit_cast(float, ~0u);
        for (int i = tid; i < (int)(sizeof(lds) / 4); i += NT)
            reinterpret_cast<uint32_t*>(lds)[i] = ~0u;
        __syncthreads();
    }
    const int nbh = p.batch * p.hq;
    const int w = blockIdx.x;
    const int qt = p.q_order ? w / nbh : p.num_q_tiles - 1 - w / nbh;
    const int b = (w % nbh) / p.hq, hq = (w % nbh) % p.hq;

    int lq, lk;
    int64_t qrow0 = 0, krow0 = 0;
    if (p.cu_q) {
        qrow0 = p.cu_q[b];
        lq = p.cu_q[b + 1] - (int)qrow0;
        krow0 = p.cu_k[b];
        lk = p.cu_k[b + 1] - (int)krow0;
    } else {
        lq = p.seqlen_q;
        lk = p.seqlen_k;
    }
    const int q0 = qt * BM;
    if (q0 >= lq) return;  // whole workgroup
    const int hkv = hq / p.group;
    const float* qb = static_cast<const float*>(p.q);
    const float* kb = static_cast<const float*>(p.k);
    const float* vb = static_cast<const float*>(p.v);
    float* ob = static_cast<float*>(p.o);
    int64_t qoff, koff, voff, ooff;
    if (p.cu_q) {
        qoff = qrow0 * p.sq_s + (int64_t)hq * p.sq_h;
        ooff = qrow0 * p.so_s + (int64_t)hq * p.so_h;
        koff = krow0 * p.sk_s + (int64_t)hkv * p.sk_h;
        voff = krow0 * p.sv_s + (int64_t)hkv * p.sv_h;
    } else {
        qoff = (int64_t)b * p.sq_b + (int64_t)hq * p.sq_h;
        ooff = (int64_t)b * p.so_b + (int64_t)hq * p.so_h;
        koff = (int64_t)b * p.sk_b + (int64_t)hkv * p.sk_h;
        voff = (int64_t)b * p.sv_b + (int64_t)hkv * p.sv_h;
    }

    // Q rows into LDS, all four waves cooperating.
    for (int e = tid; e < BM * (D / 4); e += NT) {
        const int r = e / (D / 4), c = e % (D / 4);
        f32x4 x = {0.f, 0.f, 0.f, 0.f};
        if (q0 + r < lq) x = *reinterpret_cast<const f32x4*>(qb + qoff + (int64_t)(q0 + r) * p.sq_s + 4 * c);
        *reinterpret_cast<f32x4*>(&qs[r][4 * c]) = x;
    }
    __syncthreads();

    const int qi = q0 + lane;  // every wave covers the same 64 rows
    // this sequence's index-mask layout (one shared by all when the stride is 0)
    const int32_t* gtok = p.gtok ? p.gtok + (int64_t)b * p.gtok_stride : nullptr;
    const int32_t* seg = p.seg ? p.seg + (int64_t)b * p.seg_stride : nullptr;
    RowVis rv = {0, 1, 0};
    int t_lo, t_hi;  // key tiles visited
    if constexpr (GEN) {
        if (qi < lq)
            rv = gtok ? row_vis_listed(p.band, gtok, p.num_global, qi, lq, lk)
                      : row_visibility(p.mask_kind, p.band, p.num_global, seg, p.num_seg,
                                       p.query_start, qi, lq, lk);
        const bool any = rv.pfx > 0 || rv.jlo <= rv.jhi;
        const int first = any ? (rv.pfx > 0 ? 0 : rv.jlo) : 0x3fffffff;
        const int last = any ? (rv.jlo <= rv.jhi ? rv.jhi : rv.pfx - 1) : -1;
        t_lo = __builtin_amdgcn_readfirstlane(wave_min(first)) / BN;
        t_hi = __builtin_amdgcn_readfirstlane(wave_max(last));
        t_hi = t_hi < 0 ? t_lo : t_hi / BN + 1;
    } else {
        if (qi < lq) band_row(p.band, qi, lq, lk, &rv.jlo, &rv.jhi);
        const TilePlan gp = plan_tiles(p.band, q0, BM, lq, lk, BN);
        t_lo = gp.lo;
        t_hi = gp.hi;
    }
    const int ip = qi + (lk - lq);
    // relative-position reference (see score_u): first visible key for softmax
    int jref = SOFTMAX ? (rv.pfx > 0 ? 0 : rv.jlo) : ip;
    if (GEN && SOFTMAX && gtok) {  // the smallest visible key may be one of G
        int jr = rv.jlo <= rv.jhi ? rv.jlo : 0x7fffffff;
        if (p.num_global > 0 && gtok[0] < lk) jr = min(jr, gtok[0]);
        jref = jr == 0x7fffffff ? 0 : jr;
    }
    float bias_abs = 0.0f, bias_lin = 0.0f;
    if constexpr (BIAS == kBiasAlibi || BIAS == kBiasGeneral)
        if (p.slopes) bias_abs = -p.slopes[hq] * p.unit;
    if constexpr (BIAS == kBiasRelPos || BIAS == kBiasGeneral)
        if (p.relpos) bias_lin = p.unit;
    constexpr bool MODS = SOFTCAP || BIAS != kBiasNone;
    float o[D];
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] = 0.0f;
    float m_run = -__builtin_inff(), l_run = 0.0f;

    // This wave's K and V tiles; only this wave touches them, so ordering its
    // own LDS writes and reads needs a fence, not a workgroup barrier.
    float (*ks)[D] = reinterpret_cast<float (*)[D]>(lds + wave * 2 * BN * D * 4);
    float (*vs)[D] = reinterpret_cast<float (*)[D]>(lds + (wave * 2 + 1) * BN * D * 4);
    // Scores, mask, online softmax and P V for the BN keys in ks / vs; key t
    // of the tile sits at position jpos(t) and is visible iff vis(t).
    auto consume = [&](auto jpos, auto vis) __attribute__((always_inline)) {
        float s[BN];
#pragma unroll
        for (int j = 0; j < BN; ++j) s[j] = 0.0f;
#pragma unroll
        for (int c = 0; c < D / 4; ++c) {
            f32x4 qx = *reinterpret_cast<const f32x4*>(&qs[lane][4 * c]);
#pragma unroll
            for (int j = 0; j < BN; ++j) {
                f32x4 kx = *reinterpret_cast<const f32x4*>(&ks[j][4 * c]);
                s[j] = __builtin_fmaf(qx[0], kx[0], s[j]);
                s[j] = __builtin_fmaf(qx[1], kx[1], s[j]);
                s[j] = __builtin_fmaf(qx[2], kx[2], s[j]);
                s[j] = __builtin_fmaf(qx[3], kx[3], s[j]);
            }
        }
        float mx = -__builtin_inff();
#pragma unroll
        for (int j = 0; j < BN; ++j) {
            float x = MODS ? score_u<SOFTCAP, BIAS>(s[j], p.scale_u, p.softcap_pre, p.softcap_post_u,
                                                    bias_abs, bias_lin, ip, jref, jpos(j))
                           : s[j] * p.scale_u;
            if (!vis(j)) x = -__builtin_inff();
            s[j] = x;
            mx = __builtin_fmaxf(mx, x);
        }
        float alpha = 1.0f, m_new = m_run, m_use = 0.0f;
        if constexpr (SOFTMAX) {
            // A row that has seen no key yet (m_run = -inf) and sees none of
            // this tile either (a gathered tile of global keys all inside its
            // band or past the end) keeps m = -inf with O and l at 0: the
            // exponentials take 0 in place of the max, where
            // exp2(-inf - (-inf)) would be NaN.
            m_new = __builtin_fmaxf(m_run, mx);
            m_use = m_new == -__builtin_inff() ? 0.0f : m_new;
            alpha = __builtin_amdgcn_exp2f(m_run - m_use);  // 0 when only m_run = -inf
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int d = 0; d < D; ++d) o[d] *= alpha;
        }
#pragma unroll
        for (int j = 0; j < BN; ++j) {
            float pe;
            if constexpr (SOFTMAX) {
                pe = __builtin_amdgcn_exp2f(s[j] - m_use);
                l_run += pe;
            } else {
                pe = activation<NORM>(s[j]);  // the 1/L comes at the end
            }
#pragma unroll
            for (int c = 0; c < D / 4; ++c) {
                f32x4 vx = *reinterpret_cast<const f32x4*>(&vs[j][4 * c]);
                o[4 * c + 0] = __builtin_fmaf(pe, vx[0], o[4 * c + 0]);
                o[4 * c + 1] = __builtin_fmaf(pe, vx[1], o[4 * c + 1]);
                o[4 * c + 2] = __builtin_fmaf(pe, vx[2], o[4 * c + 2]);
                o[4 * c + 3] = __builtin_fmaf(pe, vx[3], o[4 * c + 3]);
            }
        }
    };
    // K and V rows at positions key(r) (r < BN) into this wave's tiles; rows at
    // or past the sequence end are zero.
    auto stage = [&](auto key) __attribute__((always_inline)) {
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");  // previous tile fully read
#pragma unroll
        for (int i = 0; i < BN * D / 4 / 64; ++i) {
            int e = i * 64 + lane;
            int r = e / (D / 4), c = e % (D / 4);
            const int j = key(r);
            f32x4 kx = {0.f, 0.f, 0.f, 0.f}, vx = {0.f, 0.f, 0.f, 0.f};
            if (j < lk) {
                kx = *reinterpret_cast<const f32x4*>(kb + koff + (int64_t)j * p.sk_s + 4 * c);
                vx = *reinterpret_cast<const f32x4*>(vb + voff + (int64_t)j * p.sv_s + 4 * c);
            }
            *reinterpret_cast<f32x4*>(&ks[r][4 * c]) = kx;
            *reinterpret_cast<f32x4*>(&vs[r][4 * c]) = vx;
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");  // tile written
    };
    for (int kt = t_lo + wave; kt < t_hi; kt += NW) {
        const int j0 = kt * BN;
        stage([&](int r) { return j0 + r; });
        const bool band_hit = rv.jlo <= rv.jhi && rv.jhi >= j0 && rv.jlo <= j0 + BN - 1;
        if (!band_hit && j0 >= rv.pfx) continue;  // row sees none of the tile
        const bool full = j0 + BN <= rv.pfx || (rv.jlo <= j0 && j0 + BN - 1 <= rv.jhi);
        consume([&](int j) { return j0 + j; }, [&](int j) { return full || row_sees(rv, j0 + j); });
    }
    // A listed global set (global sliding window): its keys outside the row's
    // band, BN list entries per tile, the waves taking turns.
    if (GEN && gtok) {
        const int ng = p.num_global;
        for (int g0 = wave * BN; g0 < ng; g0 += NW * BN) {
            auto key = [&](int r) { return g0 + r < ng ? min(gtok[g0 + r], lk) : lk; };
            stage(key);
            consume(key, [&](int j) {
                const int kj = key(j);
                return qi < lq && kj < lk && !(kj >= rv.jlo && kj <= rv.jhi);
            });
        }
    }

    // Merge the four partial results: waves 1 and 3 into 0 and 2, then 2 into 0.
    // A partial (m, l, O) with m = -inf saw no key and contributes nothing.
    float* mb = reinterpret_cast<float*>(lds);
    auto publish = [&](int slot) {
        float* row = mb + (slot * BM + lane) * (D + 2);
#pragma unroll
        for (int d = 0; d < D; ++d) row[d] = o[d];
        row[D] = m_run;
        row[D + 1] = l_run;
    };
    auto absorb = [&](int slot) {
        const float* row = mb + (slot * BM + lane) * (D + 2);
        if constexpr (SOFTMAX) {
            const float m_o = row[D], l_o = row[D + 1];
            const float m_new = __builtin_fmaxf(m_run, m_o);
            const float a = m_run == -__builtin_inff() ? 0.0f : __builtin_amdgcn_exp2f(m_run - m_new);
            const float c = m_o == -__builtin_inff() ? 0.0f : __builtin_amdgcn_exp2f(m_o - m_new);
            m_run = m_new;
            l_run = a * l_run + c * l_o;
#pragma unroll
            for (int d = 0; d < D; ++d) o[d] = a * o[d] + c * row[d];
        } else {
#pragma unroll
            for (int d = 0; d < D; ++d) o[d] += row[d];
        }
    };
    __syncthreads();  // every wave is done with its K/V tiles
    if (wave == 1) publish(0);
    if (wave == 3) publish(1);
    __syncthreads();
    if (wave == 0) absorb(0);
    if (wave == 2) absorb(1);
    __syncthreads();
    if (wave == 2) publish(0);
    __syncthreads();
    if (wave != 0) return;
    absorb(0);

    if (qi < lq) {
        float inv;
        if constexpr (SOFTMAX)
            inv = l_run > 0.0f ? 1.0f / l_run : 0.0f;
        else
            inv = lk > 0 ? 1.0f / (float)lk : 0.0f;
        float* dst = ob + ooff + (int64_t)qi * p.so_s;
#pragma unroll
        for (int c = 0; c < D / 4; ++c) {
            f32x4 x = {o[4 * c] * inv, o[4 * c + 1] * inv, o[4 * c + 2] * inv, o[4 * c + 3] * inv};
            *reinterpret_cast<f32x4*>(dst + 4 * c) = x;
        }
        if (SOFTMAX && p.lse) {
            float lse = -__builtin_inff();
            if (l_run > 0.0f) {
                lse = (m_run + __builtin_log2f(l_run)) * kLn2;
                if (bias_lin != 0.0f) lse += (float)(ip - jref);
            }
            int64_t idx = p.cu_q ? (int64_t)hq * p.total_q + qrow0 + qi
                                 : ((int64_t)b * p.hq + hq) * lq + qi;
            p.lse[idx] = lse;
        }
    }
}

template <int D, bool SOFTCAP, int BIAS, int NORM, bool GEN>
hipError_t launch(const AttnParams& p, hipStream_t stream)
{
    int64_t blocks = (int64_t)p.num_q_tiles * p.hq * p.batch;
    hipLaunchKernelGGL((attn_fwd_f32_kernel<D, SOFTCAP, BIAS, NORM, GEN>), dim3((unsigned)blocks),
                       dim3(NT), 0, stream, p);
    return hipGetLastError();
}

template <int D, bool SOFTCAP>
hipError_t launch_d(const AttnParams& p, hipStream_t stream)
{
    const bool closed = p.mask_kind >= 0 && p.mask_kind <= 3;  // band masks of plan.h
    const bool al = p.slopes != nullptr, rp = p.relpos != 0;
    if (p.norm == kNormSoftmax && closed && !(al && rp)) {
        if (al) return launch<D, SOFTCAP, kBiasAlibi, kNormSoftmax, false>(p, stream);
        if (rp) return launch<D, SOFTCAP, kBiasRelPos, kNormSoftmax, false>(p, stream);
        return launch<D, SOFTCAP, kBiasNone, kNormSoftmax, false>(p, stream);
    }
    const bool bias = al || rp;
    if (p.norm == kNormRelu)
        return bias ? launch<D, SOFTCAP, kBiasGeneral, kNormRelu, true>(p, stream)
                    : launch<D, SOFTCAP, kBiasNone, kNormRelu, true>(p, stream);
    if (p.norm == kNormSigmoid)
        return bias ? launch<D, SOFTCAP, kBiasGeneral, kNormSigmoid, true>(p, stream)
                    : launch<D, SOFTCAP, kBiasNone, kNormSigmoid, true>(p, stream);
    return bias ? launch<D, SOFTCAP, kBiasGeneral, kNormSoftmax, true>(p, stream)
                : launch<D, SOFTCAP, kBiasNone, kNormSoftmax, true>(p, stream);
}

}  // namespace

int f32_block_m() { return BM; }

hipError_t launch_f32(const AttnParams& p, int head_dim, hipStream_t stream)
{
    const bool sc = p.softcap > 0.0f;
    if (head_dim == 128) return sc ? launch_d<128, true>(p, stream) : launch_d<128, false>(p, stream);
    return sc ? launch_d<64, true>(p, stream) : launch_d<64, false>(p, stream);
}

}  // namespace attn

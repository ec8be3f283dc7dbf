/*
 * attn_ref.c -- CPU oracle for the attention forward pass.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
 * calls this file; only the test-suite, the smoke check and the benchmark's
 * CPU-baseline leg do. It shares no code, header or table with the HIP path.
 *
 * What it computes: for every requested query row, the plain definition of
 * scaled-dot-product attention written out in fp64 with every score
 * materialised (no tiling, no online softmax, no reordering):
 *
 *   Eq. 1 (Section 2.2):  O = Softmax(Q K^T / sqrt(d)) V
 *   Eq. 2 / Appendix A:   O = Norm(Mask(Score(S))) V, with the raw score
 *                         S_ij = scale * q_i . k_j  (Appendix A, "Score
 *                         Modifications"), mask entries 0 = visible and
 *                         -inf = masked (Appendix A, preamble), Norm = softmax.
 *   Softcap (Appendix A, "Softcap Attention"):  Score(S) = C tanh(S / C).
 *   Relative position (Appendix A, "Relative Position Embeddings"):
 *                         Score(S) = S + (i - j).
 *   Masks (Appendix A, "Mask Variants"): PrefixLM, Global Sliding Window,
 *                         Share Question Mask, Causal Blockwise Mask, each
 *                         written as its printed case analysis.
 *   Norm (Appendix A, "Normalization Variants"): softmax, or
 *                         Norm(S) = ReLU(S) / L, or Sigmoid(S) / L, with L the
 *                         key sequence length.
 *
 * Readings taken where the paper names a variant without defining it
 * (Appendix C and E name causal, sliding window and ALiBi only):
 *   - order of score modifications: scale, then softcap, then ALiBi bias,
 *     then the mask;
 *   - ALiBi bias = -slope_h * |i + (Lk - Lq) - j|, slope given per query head;
 *   - causal: key j visible iff j <= i + (Lk - Lq) (bottom-right aligned);
 *   - sliding window: visible iff (i + Lk - Lq) - j <= window_left and
 *     j - (i + Lk - Lq) <= window_right, a negative bound meaning unbounded;
 *   - grouped-query heads: kv head = q head / (Hq / Hkv);
 *   - variable length: sequence s owns rows cu[s] .. cu[s+1]-1; sequences
 *     never see each other;
 *   - LSE = natural log of the sum of exp over visible final scores;
 *   - a row with no visible key gets O = 0 and LSE = -inf;
 *   - PrefixLM: positions are 0-based and the prefix of length L_p is keys
 *     0 .. L_p-1, so j < L_p is visible to every row, else causal;
 *   - relative position and ALiBi use the key-axis query position
 *     i' = i + (Lk - Lq) and are added after the soft-cap;
 *   - Global Sliding Window: |i' - j| <= w is taken as the two window bounds
 *     (window_left = window_right = w in the paper's form); G is any set of
 *     key-axis positions given as a list;
 *   - Share Question: every key position carries a segment id, -1 for the
 *     prompt Q and k >= 0 for response A_k;
 *   - Causal Blockwise: every key position carries its document id D_j and
 *     rows at key-axis positions >= L_q are the test query;
 *   - ReLU / Sigmoid: L = Lk of the row's sequence; masked scores are -inf,
 *     which both activations send to 0; there is no LSE (NaN is written).
 *
 * Inputs are fp32 arrays holding the exact values of the bf16 or fp32 inputs;
 * every operation on them is in fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct ref_params {
    int32_t batch;        /* B, or number of sequences when varlen            */
    int32_t hq, hkv;      /* query heads, key/value heads (hq % hkv == 0)      */
    int32_t sq, sk;       /* fixed-length query / key length (ignored varlen)  */
    int32_t d;            /* head dimension                                    */
    double scale;         /* multiplies q . k                                  */
    int32_t mask_kind;    /* 0 none, 1 causal, 2 sliding window, 3 PrefixLM,
                             4 global sliding window, 5 share question,
                             6 causal blockwise                                */
    int32_t window_left;  /* sliding window: max (i' - j), < 0 = unbounded     */
    int32_t window_right; /* sliding window: max (j - i'), < 0 = unbounded     */
    const double *slopes; /* ALiBi slope per query head, or NULL               */
    double softcap;       /* C > 0 enables C tanh(S / C)                       */
    const int32_t *cu_q;  /* varlen: int32[batch+1] query prefix sums, or NULL */
    const int32_t *cu_k;  /* varlen: int32[batch+1] key prefix sums, or NULL   */
    int32_t prefix_len;   /* PrefixLM: prefix length L_p                        */
    int32_t relpos;       /* 1: Score(S) = S + (i' - j)                          */
    int32_t norm_kind;    /* 0 softmax, 1 ReLU(S)/L, 2 Sigmoid(S)/L              */
    const int32_t *token_ids; /* share question / blockwise: id per key position */
    int32_t query_start;  /* causal blockwise: first test-query position L_q    */
    const int32_t *global_tokens; /* global sliding window: the positions of G  */
    int32_t num_global;   /* number of entries in global_tokens                 */
} ref_params;

static int in_global(const ref_params *p, int64_t pos)
{
    for (int32_t g = 0; g < p->num_global; ++g)
        if (p->global_tokens[g] == pos) return 1;
    return 0;
}

/* Is key j visible from query row i of a sequence with Lq queries and Lk keys? */
static int visible(const ref_params *p, int64_t i, int64_t j, int64_t lq, int64_t lk)
{
    int64_t ii = i + (lk - lq); /* query position on the key axis */
    (void)lq;
    if (j < 0 || j >= lk) return 0;
    if (p->mask_kind == 0) return 1;
    if (p->mask_kind == 1) return j <= ii;
    if (p->mask_kind == 2) {
        if (p->window_left >= 0 && ii - j > p->window_left) return 0;
        if (p->window_right >= 0 && j - ii > p->window_right) return 0;
        return 1;
    }
    if (p->mask_kind == 3) { /* PrefixLM */
        if (j < p->prefix_len) return 1; /* prefix visibility */
        return j <= ii;                  /* causal generation */
    }
    if (p->mask_kind == 4) { /* Global Sliding Window */
        if (in_global(p, ii) || in_global(p, j)) return 1;
        if (p->window_left >= 0 && ii - j > p->window_left) return 0;
        if (p->window_right >= 0 && j - ii > p->window_right) return 0;
        return 1;
    }
    if (p->mask_kind == 5) { /* Share Question: prompt id -1, response A_k id k */
        if (j > ii || ii < 0) return 0;
        int32_t idi = p->token_ids[ii], idj = p->token_ids[j];
        if (idi < 0) return idj < 0;     /* prompt self-attention         */
        return idj < 0 || idj == idi;    /* response -> prompt + itself   */
    }
    if (p->mask_kind == 6) { /* Causal Blockwise */
        if (j > ii || ii < 0) return 0;
        if (ii >= p->query_start) return 1;          /* test query visibility   */
        return p->token_ids[ii] == p->token_ids[j];  /* demonstration isolation */
    }
    return 0;
}

/* Final score of pair (i, j) before masking: Score(S_ij). */
static double score(const ref_params *p, const float *qi, const float *kj,
                    int32_t h, int64_t i, int64_t j, int64_t lq, int64_t lk)
{
    double dot = 0.0;
    for (int32_t t = 0; t < p->d; ++t) dot += (double)qi[t] * (double)kj[t];
    double s = p->scale * dot;
    if (p->softcap > 0.0) s = p->softcap * tanh(s / p->softcap);
    if (p->slopes) {
        int64_t rel = i + (lk - lq) - j;
        s -= p->slopes[h] * (double)(rel < 0 ? -rel : rel);
    }
    if (p->relpos) s += (double)(i + (lk - lq) - j);
    return s;
}

/*
 * Compute O and LSE for the rows listed in `rows` (flat LSE indices), or for
 * every row when rows == NULL.
 *
 * Layouts (contiguous):
 *   fixed  : q, o [B,Hq,Sq,D]; k, v [B,Hkv,Sk,D]; lse [B,Hq,Sq]
 *   varlen : q, o [Tq,Hq,D];   k, v [Tk,Hkv,D];   lse [Hq,Tq]
 * A row's flat LSE index is (b*Hq + h)*Sq + i (fixed) or h*Tq + t (varlen).
 * probs, when not NULL (fixed length only), receives P [B,Hq,Sq,Sk].
 * Returns 0, or -1 on bad parameters / allocation failure.
 */
int attn_ref_fwd(const ref_params *p, const float *q, const float *k, const float *v,
                 double *o, double *lse, const int64_t *rows, int64_t nrows,
                 double *probs)
{
    if (!p || !q || !k || !v || !o || !lse) return -1;
    if (p->hq <= 0 || p->hkv <= 0 || p->hq % p->hkv != 0 || p->d <= 0 || p->batch < 0) return -1;
    if (p->mask_kind < 0 || p->mask_kind > 6 || p->norm_kind < 0 || p->norm_kind > 2) return -1;
    if ((p->mask_kind == 5 || p->mask_kind == 6) && !p->token_ids) return -1;
    if (p->num_global < 0 || (p->num_global > 0 && !p->global_tokens)) return -1;
    int varlen = p->cu_q != NULL;
    if (varlen && (p->cu_k == NULL || probs != NULL)) return -1;
    int64_t tq = varlen ? p->cu_q[p->batch] : 0;
    int64_t total_rows = varlen ? (int64_t)p->hq * tq : (int64_t)p->batch * p->hq * p->sq;
    if (rows == NULL) nrows = total_rows;
    int64_t max_lk = 0;
    if (varlen) {
        for (int32_t s = 0; s < p->batch; ++s) {
            int64_t lk = p->cu_k[s + 1] - p->cu_k[s];
            if (lk > max_lk) max_lk = lk;
        }
    } else {
        max_lk = p->sk;
    }
    const int32_t group = p->hq / p->hkv;
    int failed = 0;

#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)(max_lk > 0 ? max_lk : 1));
        if (!s) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 16)
        for (int64_t n = 0; n < nrows; ++n) {
            if (!s) continue;
            int64_t row = rows ? rows[n] : n;
            if (row < 0 || row >= total_rows) {
#pragma omp atomic write
                failed = 1;
                continue;
            }
            /* locate (sequence b, head h, query index i within the sequence) */
            int32_t b, h;
            int64_t i, lq, lk;
            const float *qi;
            const float *kbase, *vbase;
            int64_t kstride; /* elements between consecutive keys */
            double *oi;
            if (varlen) {
                h = (int32_t)(row / tq);
                int64_t t = row % tq;
                b = 0;
                while (p->cu_q[b + 1] <= t) ++b;
                i = t - p->cu_q[b];
                lq = p->cu_q[b + 1] - p->cu_q[b];
                lk = p->cu_k[b + 1] - p->cu_k[b];
                qi = q + (t * p->hq + h) * p->d;
                oi = o + (t * p->hq + h) * p->d;
                int32_t hk = h / group;
                kbase = k + ((int64_t)p->cu_k[b] * p->hkv + hk) * p->d;
                vbase = v + ((int64_t)p->cu_k[b] * p->hkv + hk) * p->d;
                kstride = (int64_t)p->hkv * p->d;
            } else {
                i = row % p->sq;
                h = (int32_t)((row / p->sq) % p->hq);
                b = (int32_t)(row / ((int64_t)p->sq * p->hq));
                lq = p->sq;
                lk = p->sk;
                qi = q + row * p->d;
                oi = o + row * p->d;
                int32_t hk = h / group;
                kbase = k + (((int64_t)b * p->hkv + hk) * p->sk) * p->d;
                vbase = v + (((int64_t)b * p->hkv + hk) * p->sk) * p->d;
                kstride = p->d;
            }
            /* materialise every score of the row, masked ones as -inf */
            double mx = -INFINITY;
            for (int64_t j = 0; j < lk; ++j) {
                if (visible(p, i, j, lq, lk))
                    s[j] = score(p, qi, kbase + j * kstride, h, i, j, lq, lk);
                else
                    s[j] = -INFINITY;
                if (s[j] > mx) mx = s[j];
            }
            for (int32_t t = 0; t < p->d; ++t) oi[t] = 0.0;
            if (p->norm_kind != 0) { /* act(S) / L, no running max, no LSE */
                for (int64_t j = 0; j < lk; ++j) {
                    double a;
                    if (s[j] == -INFINITY)
                        a = 0.0;
                    else if (p->norm_kind == 1)
                        a = s[j] > 0.0 ? s[j] : 0.0;
                    else
                        a = 1.0 / (1.0 + exp(-s[j]));
                    double pj = a / (double)lk;
                    if (probs) probs[row * p->sk + j] = pj;
                    const float *vj = vbase + j * kstride;
                    for (int32_t t = 0; t < p->d; ++t) oi[t] += pj * (double)vj[t];
                }
                lse[row] = NAN;
                continue;
            }
            if (mx == -INFINITY) { /* no visible key */
                lse[row] = -INFINITY;
                if (probs) for (int64_t j = 0; j < lk; ++j) probs[row * p->sk + j] = 0.0;
                continue;
            }
            double z = 0.0;
            for (int64_t j = 0; j < lk; ++j) z += exp(s[j] - mx);
            for (int64_t j = 0; j < lk; ++j) {
                double pj = exp(s[j] - mx) / z;
                if (probs) probs[row * p->sk + j] = pj;
                const float *vj = vbase + j * kstride;
                for (int32_t t = 0; t < p->d; ++t) oi[t] += pj * (double)vj[t];
            }
            lse[row] = mx + log(z);
        }
        free(s);
    }
    return failed ? -1 : 0;
}

/* Number of threads the OpenMP runtime will use for a parallel region. */
int attn_ref_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}

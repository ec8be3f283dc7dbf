// row_vis.h -- keys visible to one query row under the masks whose pattern
// depends on per-position data (Appendix A, "Mask Variants"), host and device.
//
// Every mask kind reduces, for one row, to a prefix [0, pfx) plus a band
// [jlo, jhi] of keys (either part may be empty):
//   Global Sliding Window: a row whose key-axis position i' is global sees
//     every key; any other row sees the global positions 0..G-1 plus the
//     window band.
//   Share Question: positions before the first segment start are the prompt;
//     segment k covers [s_k, s_{k+1}). A prompt row sees the prompt causally;
//     a response row sees the prompt plus its own segment up to itself.
//   Causal Blockwise: segment k is document k (positions before s_0 form one
//     more document). A row before the test query (i' < L_q) sees its own
//     document up to itself; a test-query row sees every key up to itself.
//   The closed-form kinds (none, causal, sliding window, PrefixLM) are the
//   band of plan.h with no separate prefix.
// The pair is normalised so that pfx > 0 implies pfx < jlo <= jhi (a prefix
// touching the band is merged into it).
#pragma once

#include <stdint.h>

#include "plan.h"

struct RowVis {
    int32_t pfx;       // keys j < pfx are visible
    int32_t jlo, jhi;  // keys jlo <= j <= jhi are visible (empty if jlo > jhi)
};

// Largest k with seg[k] <= pos (seg strictly increasing), or -1.
ATTN_HD int32_t segment_of(const int32_t* seg, int32_t n, int32_t pos)
{
    int32_t lo = 0, hi = n;  // answer in [lo - 1, hi - 1]
    while (lo < hi) {
        int32_t mid = (lo + hi) >> 1;
        if (seg[mid] <= pos)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo - 1;
}

// mask kinds of attn.h handled here
enum : int32_t {
    kMaskGlobalWindow = 4,
    kMaskShareQuestion = 5,
    kMaskCausalBlockwise = 6,
};

// Visible keys of query row i (0 <= i < lq) of a sequence with lk keys.
// `seg` holds the num_seg segment starts (share question, causal blockwise).
ATTN_HD RowVis row_visibility(int32_t kind, KeyBand band, int32_t num_global, const int32_t* seg,
                              int32_t num_seg, int32_t query_start, int32_t i, int32_t lq,
                              int32_t lk)
{
    RowVis r = {0, 1, 0};
    if (lk <= 0) return r;
    const int32_t ip = i + (lk - lq);
    if (kind == kMaskGlobalWindow) {
        if (ip >= 0 && ip < num_global) {
            r.jlo = 0;
            r.jhi = lk - 1;
        } else {
            band_row(band, i, lq, lk, &r.jlo, &r.jhi);
            r.pfx = num_global < lk ? num_global : lk;
        }
    } else if (kind == kMaskShareQuestion || kind == kMaskCausalBlockwise) {
        if (ip < 0) return r;  // no key at or before this row
        r.jhi = ip < lk - 1 ? ip : lk - 1;
        if (kind == kMaskCausalBlockwise && ip >= query_start) {
            r.jlo = 0;
        } else {
            int32_t k = segment_of(seg, num_seg, ip);
            r.jlo = k < 0 ? 0 : seg[k];
            if (kind == kMaskShareQuestion && k >= 0) r.pfx = seg[0] < lk ? seg[0] : lk;
        }
    } else {
        band_row(band, i, lq, lk, &r.jlo, &r.jhi);
    }
    if (r.jlo < 0) r.jlo = 0;
    if (r.pfx < 0) r.pfx = 0;
    if (r.jlo > r.jhi) {  // band empty: the prefix alone, as a band
        if (r.pfx > 0) {
            r.jlo = 0;
            r.jhi = r.pfx - 1;
        }
        r.pfx = 0;
    } else if (r.pfx >= r.jlo) {  // prefix touches the band: one interval
        r.jlo = 0;
        if (r.jhi < r.pfx - 1) r.jhi = r.pfx - 1;
        r.pfx = 0;
    }
    return r;
}

// Is key j visible under `r`?
ATTN_HD bool row_sees(RowVis r, int32_t j) { return j < r.pfx || (j >= r.jlo && j <= r.jhi); }

// Is key-axis position ip one of the sorted list g of ng positions?
ATTN_HD bool listed(const int32_t* g, int32_t ng, int32_t ip)
{
    const int32_t k = ip >= 0 ? segment_of(g, ng, ip) : -1;
    return k >= 0 && g[k] == ip;
}

// Global sliding window with G given as a sorted list g of ng positions: a row
// whose key-axis position is in G sees every key; any other row sees its
// window band here, and the keys of G outside that band are taken separately
// (they are not a prefix, so they do not fit the prefix + band form).
ATTN_HD RowVis row_vis_listed(KeyBand band, const int32_t* g, int32_t ng, int32_t i, int32_t lq,
                              int32_t lk)
{
    RowVis r = {0, 1, 0};
    if (lk <= 0) return r;
    const int32_t ip = i + (lk - lq);
    const int32_t k = ip >= 0 ? segment_of(g, ng, ip) : -1;
    if (k >= 0 && g[k] == ip) {
        r.jlo = 0;
        r.jhi = lk - 1;
    } else {
        band_row(band, i, lq, lk, &r.jlo, &r.jhi);
    }
    return r;
}

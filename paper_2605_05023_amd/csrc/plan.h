// plan.h -- key-tile planning for one block of query rows (host and device).
//
// The masks with a closed-form plan are bands on the key axis: query row i
// of a sequence with lq queries and lk keys sits at key position
// i' = i + (lk - lq) and sees keys j with lo(i) <= j <= hi(i), where
//   lo(i) = max(0, i' - window_left)   (0 when window_left < 0)
//   hi(i) = min(lk - 1, max(i' + window_right, prefix - 1))
//           (lk - 1 when window_right < 0; prefix only with lo = 0).
// No-mask is the band (-1, -1), causal is (-1, 0) and PrefixLM (Appendix A,
// "PrefixLM") is causal plus a prefix: keys j < L_p are visible to every row,
// so hi(i) = max(i', L_p - 1). Both bounds grow with i, so the keys seen by a
// run of consecutive rows form one interval and a key tile is either
// untouched, fully visible for every row, or partial.
// Splitting the key loop at those boundaries keeps the element mask out of
// the fully visible tiles and skips untouched ones (loop splitting of the
// iteration space, Section 3.4, Fig. 4; block-level skipping, Appendix C).
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define ATTN_HD __host__ __device__ __forceinline__
#else
#define ATTN_HD static inline
#endif

struct KeyBand {
    int32_t wl;  // max i' - j, < 0 = unbounded
    int32_t wr;  // max j - i', < 0 = unbounded
    int32_t pl;  // keys j < pl are visible to every row (PrefixLM); needs wl < 0
};

// Visible key interval [lo, hi] of row i (empty when lo > hi).
ATTN_HD void band_row(KeyBand b, int32_t i, int32_t lq, int32_t lk, int32_t* lo, int32_t* hi)
{
    int32_t ip = i + (lk - lq);
    int32_t l = b.wl < 0 ? 0 : ip - b.wl;
    int32_t h = b.wr < 0 ? lk - 1 : ip + b.wr;
    if (h < b.pl - 1) h = b.pl - 1;
    *lo = l < 0 ? 0 : l;
    *hi = h > lk - 1 ? lk - 1 : h;
}

struct TilePlan {
    int32_t lo;       // first key tile touched
    int32_t full_lo;  // first fully visible tile
    int32_t full_hi;  // one past the last fully visible tile
    int32_t hi;       // one past the last touched tile (hi == lo: none)
};

ATTN_HD int32_t floor_div(int32_t a, int32_t b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

// Plan for query rows [q0, q0 + rows) (rows beyond lq are ignored) against
// key tiles of bn keys.
ATTN_HD TilePlan plan_tiles(KeyBand b, int32_t q0, int32_t rows, int32_t lq, int32_t lk, int32_t bn)
{
    TilePlan p = {0, 0, 0, 0};
    int32_t r0 = q0 < 0 ? 0 : q0;
    int32_t r1 = q0 + rows - 1;
    if (r1 > lq - 1) r1 = lq - 1;
    if (rows <= 0 || r0 > r1 || lk <= 0) return p;
    int32_t lo0, hi0, lo1, hi1;
    band_row(b, r0, lq, lk, &lo0, &hi0);
    band_row(b, r1, lq, lk, &lo1, &hi1);
    // union of the rows' intervals: [lo of the first non-empty row, hi(r1)]
    int32_t jlo = lo0, jhi = hi1;
    if (jlo > jhi) return p;
    // Only rows with i' + window_right < 0 are empty (a causal block with
    // lq > lk); hi grows by one per row there, so the first non-empty row is
    // r0 - hi0 and the union starts at its lo.
    if (hi0 < lo0) {
        int32_t r = r0 - hi0;
        if (r > r1) return p;
        int32_t lo_r, hi_r;
        band_row(b, r, lq, lk, &lo_r, &hi_r);
        jlo = lo_r;
    }
    p.lo = jlo / bn;
    p.hi = jhi / bn + 1;
    // fully visible tiles: lo(r1) <= j0 and j0 + bn - 1 <= hi(r0)
    int32_t flo = (lo1 + bn - 1) / bn;
    int32_t fhi = hi0 < 0 ? 0 : (hi0 + 1) / bn;
    if (hi0 < lo0) fhi = 0;  // row r0 sees nothing: no tile is full for every row
    if (flo < p.lo) flo = p.lo;
    if (fhi > p.hi) fhi = p.hi;
    if (flo >= fhi) {
        p.full_lo = p.full_hi = p.hi;
    } else {
        p.full_lo = flo;
        p.full_hi = fhi;
    }
    return p;
}

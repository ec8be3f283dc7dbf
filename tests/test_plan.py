"""The key-tile planner (host mirror of the in-kernel one) against brute force.

Ground truth for visibility comes from the pinned CPU oracle: with zero
queries every visible key gets probability 1/n_i > 0 and every masked key 0,
so P > 0 is exactly the mask. Each tile is then classified by enumeration:
untouched (no visible pair), full (every pair visible and the tile inside the
keys) or partial, and the plan must skip exactly the untouched tiles and
mark exactly the full ones as check-free.
"""
import itertools
import random

import numpy as np
import pytest
import torch

import oracle
import paper_2605_05023_amd as attn

MASKS = [
    (attn.ATTN_MASK_NONE, -1, -1, 0),
    (attn.ATTN_MASK_CAUSAL, -1, -1, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 0, 0, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 5, 0, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 17, 3, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, -1, 9, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 40, -1, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 1023, 0, 0),
    (attn.ATTN_MASK_PREFIX_LM, -1, -1, 0),
    (attn.ATTN_MASK_PREFIX_LM, -1, -1, 1),
    (attn.ATTN_MASK_PREFIX_LM, -1, -1, 17),
    (attn.ATTN_MASK_PREFIX_LM, -1, -1, 64),
    (attn.ATTN_MASK_PREFIX_LM, -1, -1, 300),
]


def visibility(mask, wl, wr, lq, lk, prefix=0, **kw):
    q = torch.zeros((1, 1, lq, 1))
    k = torch.ones((1, 1, lk, 1))
    v = torch.ones((1, 1, lk, 1))
    _, _, p = oracle.attention(q, k, v, scale=1.0, mask=mask, window_left=wl, window_right=wr,
                               prefix_len=prefix, want_probs=True, **kw)
    return p[0, 0] > 0


def check_plan(vis, mask, wl, wr, q0, rows, bn, prefix=0):
    lq, lk = vis.shape
    lo, flo, fhi, hi = attn.plan_tiles(mask, wl, wr, q0, rows, lq, lk, bn, prefix_len=prefix)
    r1 = min(q0 + rows, lq)
    ntiles = (lk + bn - 1) // bn + 2
    assert lo <= flo <= fhi <= hi or (lo == hi and flo == fhi)
    for t in range(ntiles):
        j0, j1 = t * bn, min((t + 1) * bn, lk)
        blk = vis[q0:r1, j0:j1] if j0 < lk and q0 < r1 else np.zeros((0, 0), bool)
        touched = blk.size > 0 and blk.any()
        full = blk.size > 0 and blk.all() and (t + 1) * bn <= lk
        in_range = lo <= t < hi
        in_full = flo <= t < fhi
        assert in_range == touched, (mask, wl, wr, q0, rows, lq, lk, bn, t, (lo, flo, fhi, hi))
        assert in_full == full, (mask, wl, wr, q0, rows, lq, lk, bn, t, (lo, flo, fhi, hi))


@pytest.mark.parametrize("mask,wl,wr,prefix", MASKS)
def test_plan_matches_brute_force(mask, wl, wr, prefix):
    rng = random.Random(1234 + mask * 100 + wl + prefix)
    shapes = [(1, 1), (5, 5), (64, 64), (130, 130), (200, 77), (77, 200), (257, 300), (3, 40)]
    for lq, lk in shapes:
        vis = visibility(mask, wl, wr, lq, lk, prefix)
        for bn, rows in itertools.product((16, 32, 64), (1, 32, 128)):
            starts = sorted({0, rows, max(0, lq - rows), rng.randrange(0, max(1, lq))})
            for q0 in starts:
                if q0 < lq:
                    check_plan(vis, mask, wl, wr, q0, rows, bn, prefix)


def _ids(S, starts):
    ids = [-1] * S
    for k, st in enumerate(starts):
        for p in range(st, S):
            ids[p] = k
    return ids


# (mask, window_left, window_right, prefix_len, num_global, segment_starts, query_start)
ROW_CASES = [
    (attn.ATTN_MASK_CAUSAL, -1, -1, 0, 0, None, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 9, 2, 0, 0, None, 0),
    (attn.ATTN_MASK_PREFIX_LM, -1, -1, 23, 0, None, 0),
    (attn.ATTN_MASK_GLOBAL_SLIDING_WINDOW, 4, 4, 0, 3, None, 0),
    (attn.ATTN_MASK_GLOBAL_SLIDING_WINDOW, 0, 7, 0, 0, None, 0),
    (attn.ATTN_MASK_GLOBAL_SLIDING_WINDOW, 2, 2, 0, 50, None, 0),
    (attn.ATTN_MASK_SHARE_QUESTION, -1, -1, 0, 0, [10, 17, 40], 0),
    (attn.ATTN_MASK_SHARE_QUESTION, -1, -1, 0, 0, [0, 5], 0),
    (attn.ATTN_MASK_CAUSAL_BLOCKWISE, -1, -1, 0, 0, [0, 8, 9, 30], 35),
    (attn.ATTN_MASK_CAUSAL_BLOCKWISE, -1, -1, 0, 0, [4, 20], 0),
    (attn.ATTN_MASK_CAUSAL_BLOCKWISE, -1, -1, 0, 0, [0, 12], 100),
]


@pytest.mark.parametrize("case", ROW_CASES, ids=lambda c: f"mask{c[0]}_{c[1]}_{c[2]}_{c[3]}_{c[4]}")
def test_row_range_matches_oracle(case):
    """The kernels' per-row visible ranges (prefix + band) equal the oracle's
    mask, row by row, for every mask kind (Sq == Sk and Sq < Sk)."""
    mask, wl, wr, prefix, ng, starts, qs = case
    for lq, lk in ((47, 47), (20, 47), (1, 5)):
        kw = {}
        if starts is not None:
            kw["token_ids"] = _ids(lk, starts)
        if mask == attn.ATTN_MASK_GLOBAL_SLIDING_WINDOW:
            kw["global_tokens"] = list(range(ng))
        vis = visibility(mask, wl, wr, lq, lk, prefix, query_start=qs, **kw)
        d = attn.AttnVariantDesc.new()
        d.mask_kind, d.window_left, d.window_right = mask, wl, wr
        d.prefix_len, d.num_global, d.query_start, d.scale = prefix, ng, qs, 1.0
        d.num_segments = len(starts) if starts else 0
        for i in range(lq):
            pfx, jlo, jhi = attn.row_range(d, i, lq, lk, segment_starts=starts)
            mine = np.array([j < pfx or jlo <= j <= jhi for j in range(lk)])
            assert np.array_equal(mine, vis[i]), (case, lq, lk, i, (pfx, jlo, jhi))
            assert pfx == 0 or pfx < jlo  # normalised form the kernels rely on


def test_plan_rejects_per_row_masks():
    for mask in (attn.ATTN_MASK_GLOBAL_SLIDING_WINDOW, attn.ATTN_MASK_SHARE_QUESTION,
                 attn.ATTN_MASK_CAUSAL_BLOCKWISE):
        with pytest.raises(attn.AttnError):
            attn.plan_tiles(mask, -1, -1, 0, 128, 256, 256, 64)


def test_plan_workload_shapes():
    # causal 2048 with 128-row blocks and 64-key tiles: block t sees 2t+2 tiles, 2t full
    # (an empty full range is reported as [hi, hi))
    for t in range(16):
        expect = (0, 0, 2 * t, 2 * t + 2) if t else (0, 2, 2, 2)
        assert attn.plan_tiles(attn.ATTN_MASK_CAUSAL, -1, -1, 128 * t, 128, 2048, 2048, 64) == expect
    # window 1023 (keys i-1023..i) at S = 8192: rows 128t..128t+127 touch keys
    # 128t-1023 .. 128t+127, i.e. tiles 2t-16 .. 2t+1: at most 18 of 128 tiles
    worst = 0
    for t in range(64):
        lo, flo, fhi, hi = attn.plan_tiles(attn.ATTN_MASK_SLIDING_WINDOW, 1023, 0, 128 * t, 128,
                                           8192, 8192, 64)
        worst = max(worst, hi - lo)
    assert worst == 18


def test_plan_empty_and_offset_rows():
    # causal with lq > lk: the first lq - lk rows see nothing
    assert attn.plan_tiles(attn.ATTN_MASK_CAUSAL, -1, -1, 0, 4, 10, 3, 64) == (0, 0, 0, 0)
    lo, flo, fhi, hi = attn.plan_tiles(attn.ATTN_MASK_CAUSAL, -1, -1, 0, 10, 10, 3, 64)
    assert (lo, hi) == (0, 1) and flo == fhi
    # no keys at all
    assert attn.plan_tiles(attn.ATTN_MASK_NONE, -1, -1, 0, 8, 8, 0, 64)[0] == \
        attn.plan_tiles(attn.ATTN_MASK_NONE, -1, -1, 0, 8, 8, 0, 64)[3]

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
    (attn.ATTN_MASK_NONE, -1, -1),
    (attn.ATTN_MASK_CAUSAL, -1, -1),
    (attn.ATTN_MASK_SLIDING_WINDOW, 0, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 5, 0),
    (attn.ATTN_MASK_SLIDING_WINDOW, 17, 3),
    (attn.ATTN_MASK_SLIDING_WINDOW, -1, 9),
    (attn.ATTN_MASK_SLIDING_WINDOW, 40, -1),
    (attn.ATTN_MASK_SLIDING_WINDOW, 1023, 0),
]


def visibility(mask, wl, wr, lq, lk):
    q = torch.zeros((1, 1, lq, 1))
    k = torch.ones((1, 1, lk, 1))
    v = torch.ones((1, 1, lk, 1))
    _, _, p = oracle.attention(q, k, v, scale=1.0, mask=mask, window_left=wl, window_right=wr,
                               want_probs=True)
    return p[0, 0] > 0


def check_plan(vis, mask, wl, wr, q0, rows, bn):
    lq, lk = vis.shape
    lo, flo, fhi, hi = attn.plan_tiles(mask, wl, wr, q0, rows, lq, lk, bn)
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


@pytest.mark.parametrize("mask,wl,wr", MASKS)
def test_plan_matches_brute_force(mask, wl, wr):
    rng = random.Random(1234 + mask * 100 + wl)
    shapes = [(1, 1), (5, 5), (64, 64), (130, 130), (200, 77), (77, 200), (257, 300), (3, 40)]
    for lq, lk in shapes:
        vis = visibility(mask, wl, wr, lq, lk)
        for bn, rows in itertools.product((16, 32, 64), (1, 32, 128)):
            starts = sorted({0, rows, max(0, lq - rows), rng.randrange(0, max(1, lq))})
            for q0 in starts:
                if q0 < lq:
                    check_plan(vis, mask, wl, wr, q0, rows, bn)


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

"""GPU parity for per-sequence index-mask layouts: every sequence of a batch
(fixed length, or packed) with its own segment starts (share question,
causal blockwise) or its own listed global set (global sliding window,
Appendix A "Mask Variants"), passed as one row per sequence
(attn_variant_desc.segment_stride / global_stride). Each sequence is compared
element by element with the CPU oracle run on that sequence alone with its own
layout; a layout repeated in every row must give exactly the shared layout's
result. Both head dims, grouped-query heads, the three normalisations and
fp32 are covered; ATTN_FLAG_VALIDATE checks every row on the host.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import LSE_TOL, O_TOL, gpu_available, log
from paper_2605_05023_amd import fwd
from paper_2605_05023_amd.workloads import (MASK_CAUSAL_BLOCKWISE, MASK_GLOBAL_WINDOW, MASK_NAMES,
                                            MASK_SHARE_QUESTION, alibi_slopes)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]
DEV = "cuda:0"


def _token_ids(starts, n):
    """Oracle segment id per key position: the largest k with start_k <= pos
    (-1 before the first start)."""
    ids = [-1] * n
    for k, st in enumerate(starts):
        for pos in range(st, n):
            ids[pos] = k
    return ids


# (name, mask, lengths (lq = lk per sequence), varlen, D, hq, hkv, dtype, norm,
#  per-sequence rows, extra)
CASES = [
    ("sq_fixed_d128", MASK_SHARE_QUESTION, [300, 300, 300], False, 128, 4, 2, "bf16", "softmax",
     [[40, 100, 220], [120, 121, 299], [0, 150, 290]], {}),
    ("sq_varlen_d64", MASK_SHARE_QUESTION, [77, 260, 301], True, 64, 2, 2, "bf16", "softmax",
     [[10, 30, 60], [100, 180, 259], [200, 320, 330]], {}),
    ("cb_fixed_d64", MASK_CAUSAL_BLOCKWISE, [257, 257], False, 64, 4, 4, "bf16", "softmax",
     [[0, 64, 65, 200], [30, 31, 129, 130]], dict(query_start=180)),
    ("cb_varlen_d128_gqa", MASK_CAUSAL_BLOCKWISE, [150, 333, 64], True, 128, 8, 2, "bf16",
     "softmax", [[20, 70, 140], [100, 250, 300], [10, 11, 63]], dict(query_start=120)),
    ("cb_varlen_sigmoid", MASK_CAUSAL_BLOCKWISE, [200, 90], True, 128, 2, 2, "bf16", "sigmoid",
     [[50, 120], [40, 80]], dict(query_start=100)),
    ("gw_fixed_d128", MASK_GLOBAL_WINDOW, [400, 400, 400], False, 128, 4, 2, "bf16", "softmax",
     [[0, 5, 200, 399], [3, 100, 250, 600], [1, 2, 3, 350]], dict(window=(32, 32))),
    ("gw_varlen_d64", MASK_GLOBAL_WINDOW, [130, 290, 45], True, 64, 4, 4, "bf16", "softmax",
     [[0, 64, 129], [7, 150, 289], [44, 60, 80]], dict(window=(16, 0))),
    ("gw_fixed_relu", MASK_GLOBAL_WINDOW, [260, 260], False, 128, 2, 2, "bf16", "relu",
     [[0, 130, 259], [60, 61, 62]], dict(window=(20, 20))),
    ("sq_fixed_fp32", MASK_SHARE_QUESTION, [150, 150], False, 64, 2, 2, "fp32", "softmax",
     [[30, 70], [100, 140]], {}),
    ("gw_varlen_fp32", MASK_GLOBAL_WINDOW, [100, 170], True, 128, 2, 1, "fp32", "softmax",
     [[0, 50, 99], [20, 21, 300]], dict(window=(10, 10))),
]


def _run(c, rows_layout, shared=None):
    name, mask, lens, varlen, D, hq, hkv, dtype, norm, rows, extra = c
    g = torch.Generator().manual_seed(sum(map(ord, name)))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    B = len(lens)
    if varlen:
        qs, ks = (sum(lens), hq, D), (sum(lens), hkv, D)
    else:
        qs, ks = (B, hq, lens[0], D), (B, hkv, lens[0], D)
    sigma = 1.5 if (extra.get("alibi") or extra.get("softcap")) else 1.0
    q = (torch.randn(qs, generator=g) * sigma).to(tdt)
    k = (torch.randn(ks, generator=g) * sigma).to(tdt)
    v = torch.randn(ks, generator=g).to(tdt)
    kw = dict(mask=MASK_NAMES[mask], norm=norm, query_start=extra.get("query_start", 0),
              softcap=extra.get("softcap", 0.0), relative_position=extra.get("relpos", False))
    if extra.get("alibi"):
        kw["alibi_slopes"] = alibi_slopes(hq).to(DEV)
    if "window" in extra:
        kw["window"] = extra["window"]
    cu = None
    if varlen:
        cu = torch.tensor([0] + list(np.cumsum(lens)), dtype=torch.int32)
        kw.update(cu_seqlens_q=cu.to(DEV), cu_seqlens_k=cu.to(DEV), max_seqlen_q=max(lens),
                  max_seqlen_k=max(lens))
    arr = torch.tensor(rows_layout if shared is None else shared, dtype=torch.int32, device=DEV)
    if mask == MASK_GLOBAL_WINDOW:
        kw["global_tokens"] = arr
    else:
        kw["segment_starts"] = arr
    res = fwd(q.to(DEV), k.to(DEV), v.to(DEV), validate=True, **kw)
    torch.cuda.synchronize()
    o, lse = res if isinstance(res, tuple) else (res, None)
    return q, k, v, cu, o, lse


def _draw_random(n=24, seed=5023):
    """Seeded random per-sequence cases: index mask, fixed or packed lengths,
    per-sequence rows (some entries at or past the sequence end), head dim,
    group size, dtype, normalisation, ALiBi, relative position, soft-cap."""
    rng = np.random.default_rng(seed)
    masks = [MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE, MASK_GLOBAL_WINDOW]
    out = []
    for i in range(n):
        mask = masks[i % 3]
        varlen = bool(rng.random() < 0.5)
        nseq = int(rng.integers(2, 5))
        lens = [int(rng.integers(1, 350)) for _ in range(nseq)] if varlen else \
            [int(rng.integers(1, 350))] * nseq
        cnt = int(rng.integers(1, 6))
        rows = []
        for L in lens:  # strictly increasing, within [0, L + 40)
            rows.append(sorted(rng.choice(L + 40, size=cnt, replace=False).tolist()))
        extra = {}
        if mask == MASK_GLOBAL_WINDOW:
            extra["window"] = (int(rng.integers(0, 60)), int(rng.choice([0, int(rng.integers(0, 60))])))
        if mask == MASK_CAUSAL_BLOCKWISE:
            extra["query_start"] = int(rng.integers(0, max(lens) + 1))
        extra["alibi"] = bool(rng.random() < 0.25)
        extra["relpos"] = bool(rng.random() < 0.2)
        extra["softcap"] = float(rng.choice([0.0, 0.0, 0.0, 30.0, 400.0]))
        dtype = "fp32" if rng.random() < 0.2 else "bf16"
        norm = str(rng.choice(["softmax"] * 4 + ["relu", "sigmoid"]))
        D = int(rng.choice([64, 128]))
        group = int(rng.choice([1, 2, 4]))
        hkv = int(rng.integers(1, 3))
        name = (f"rnd{seed}_{i:02d}_{MASK_NAMES[mask]}_{'varlen' if varlen else 'fixed'}_{dtype}"
                f"_d{D}_g{group}_{norm}")
        out.append((name, mask, lens, varlen, D, group * hkv, hkv, dtype, norm, rows, extra))
    return out


RANDOM = _draw_random()


@pytest.mark.parametrize("c", RANDOM, ids=[c[0] for c in RANDOM])
def test_per_sequence_layout_random(c):
    log(f"[parity per-sequence layout, random] {c[0]} lengths={c[2]} rows={c[9]} extra={c[10]}")
    _check(c, c[9], *_run(c, c[9]))


@pytest.mark.parametrize("c", CASES, ids=[c[0] for c in CASES])
def test_per_sequence_layout(c):
    log(f"[parity per-sequence layout] {c[0]} lengths={c[2]} rows={c[9]}")
    _check(c, c[9], *_run(c, c[9]))


# A listed global set whose keys all lie inside a row's band or past its
# sequence's end leaves that row's gathered tile fully masked; in the fp32
# kernel a wave that had not yet seen a key of the row made NaN of it
# (exp2(-inf - (-inf))). Shared layouts, every row compared with the oracle.
ALL_MASKED_GATHER = [
    ("gw_shared_fp32", MASK_GLOBAL_WINDOW, [100, 170], True, 128, 2, 1, "fp32", "softmax",
     [20, 21, 300], dict(window=(10, 10))),
    ("gw_shared_bf16", MASK_GLOBAL_WINDOW, [100, 170], True, 128, 2, 1, "bf16", "softmax",
     [20, 21, 300], dict(window=(10, 10))),
    ("gw_shared_fp32_fixed_d64", MASK_GLOBAL_WINDOW, [170, 170], False, 64, 2, 2, "fp32",
     "softmax", [20, 21, 170], dict(window=(10, 10))),
]


@pytest.mark.parametrize("c", ALL_MASKED_GATHER, ids=[c[0] for c in ALL_MASKED_GATHER])
def test_listed_global_fully_masked_gather(c):
    log(f"[parity listed global set, fully masked gather] {c[0]} G={c[9]}")
    _check(c, [c[9]] * len(c[2]), *_run(c, None, shared=c[9]))


def _check(c, rows, q, k, v, cu, o, lse):
    name, mask, lens, varlen, D, hq, hkv, dtype, norm, _, extra = c
    og = o.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(og).all()
    lg = lse.cpu().numpy().astype(np.float64) if lse is not None else None
    o_err = l_err = 0.0
    tol = O_TOL[dtype]
    for s, layout in enumerate(rows):
        if varlen:
            a, b = int(cu[s]), int(cu[s + 1])
            qs_, ks_, vs_ = q[a:b][None].transpose(1, 2), k[a:b][None].transpose(1, 2), \
                v[a:b][None].transpose(1, 2)
            o_s = og[a:b].transpose(1, 0, 2)
            l_s = lg[:, a:b] if lg is not None else None
        else:
            qs_, ks_, vs_ = q[s:s + 1], k[s:s + 1], v[s:s + 1]
            o_s = og[s]
            l_s = lg[s] if lg is not None else None
        n = ks_.shape[2]
        okw = dict(query_start=extra.get("query_start", 0),
                   norm={"softmax": 0, "relu": 1, "sigmoid": 2}[norm],
                   softcap=extra.get("softcap", 0.0), relpos=extra.get("relpos", False),
                   slopes=alibi_slopes(hq) if extra.get("alibi") else None)
        wl_, wr_ = extra.get("window", (-1, -1))
        if mask == MASK_GLOBAL_WINDOW:
            okw["global_tokens"] = list(layout)
        else:
            okw["token_ids"] = _token_ids(layout, max(n, 1))
        o_ref, lse_ref = oracle.attention(qs_.contiguous(), ks_.contiguous(), vs_.contiguous(),
                                          scale=D ** -0.5, mask=mask, window_left=wl_,
                                          window_right=wr_, **okw)
        err = float(np.abs(o_s - o_ref[0]).max())
        if norm != "softmax":
            bar = tol * float(np.abs(o_ref).max())
            assert err <= bar, (s, err, bar)
        else:
            o_err = max(o_err, err)
            inf_ref = np.isinf(lse_ref[0])
            assert np.array_equal(np.isinf(l_s), inf_ref), s
            if (~inf_ref).any():
                l_err = max(l_err, float(np.abs(l_s[~inf_ref] - lse_ref[0][~inf_ref]).max()))
    log(f"  max|dO| = {o_err:.3e} (tol {tol:.0e}), max|dLSE| = {l_err:.3e}")
    assert o_err <= tol and l_err <= LSE_TOL


@pytest.mark.parametrize("c", [CASES[0], CASES[3], CASES[5], CASES[9]],
                         ids=[c[0] for c in (CASES[0], CASES[3], CASES[5], CASES[9])])
def test_repeated_rows_equal_shared_layout(c):
    """One row per sequence, all equal, gives exactly the shared layout's output."""
    name, rows = c[0], c[9]
    log(f"[per-sequence layout = shared] {name}")
    rep = [rows[0]] * len(rows)
    *_, o1, l1 = _run(c, rep)
    *_, o2, l2 = _run(c, rep, shared=rows[0])
    assert torch.equal(o1, o2)
    if l1 is not None:
        assert torch.equal(l1, l2)

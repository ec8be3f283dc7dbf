"""GPU parity on seeded random problems whose query and key lengths differ.

Decode (one query against a key cache), chunked prefill (a query chunk
against a longer key history), more queries than keys (rows that see no key
under the bottom-right aligned masks), fixed length and packed sequences with
their own query and key lengths, across every mask kind, ALiBi, the relative
position term, the soft-cap and the three normalisations. Query i of a
sequence with Lq queries and Lk keys sits at key position i + Lk - Lq for
every variant; the oracle's reading of that is pinned on the CPU. Each case
compares every output element with the oracle at the bars of the other
parity tests.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import LSE_TOL, O_TOL, gpu_available, log
from paper_2605_05023_amd import fwd
from paper_2605_05023_amd.workloads import (MASK_CAUSAL, MASK_CAUSAL_BLOCKWISE, MASK_GLOBAL_WINDOW,
                                            MASK_NAMES, MASK_NONE, MASK_PREFIX_LM,
                                            MASK_SHARE_QUESTION, MASK_SLIDING_WINDOW, alibi_slopes)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

MASKS = [MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW, MASK_PREFIX_LM, MASK_GLOBAL_WINDOW,
         MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE]
SHAPES = ["decode", "chunked_prefill", "more_queries", "packed"]


def _lengths(rng, shape):
    """(lq, lk) per sequence for the shape family."""
    n = int(rng.integers(1, 4)) if shape != "packed" else int(rng.integers(2, 6))
    out = []
    for _ in range(n):
        lk = int(rng.integers(1, 400))
        if shape == "decode":
            out.append((1, lk))
        elif shape == "chunked_prefill":
            out.append((int(rng.integers(1, lk + 1)), lk))
        elif shape == "more_queries":
            out.append((lk + int(rng.integers(1, 100)), lk))
        else:
            out.append((int(rng.integers(0, 300)), int(rng.integers(0, 400))))
    return out


def _draw(n=40, seed=4411):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        shape = SHAPES[i % len(SHAPES)]
        lens = _lengths(rng, shape)
        varlen = shape == "packed" or rng.random() < 0.3
        if not varlen:  # one (lq, lk) for every batch entry
            lens = [lens[0]] * len(lens)
        mask = MASKS[int(rng.integers(0, len(MASKS)))]
        maxk = max(lk for _, lk in lens)
        kw = {}
        if mask in (MASK_SLIDING_WINDOW, MASK_GLOBAL_WINDOW):
            kw["window"] = (int(rng.choice([-1, int(rng.integers(0, 150))])),
                            int(rng.choice([-1, 0, int(rng.integers(0, 40))])))
            if mask == MASK_GLOBAL_WINDOW:
                kw["num_global"] = int(rng.integers(0, 12))
                g = np.random.default_rng(kw["num_global"] * 7919 + i)
                if g.random() < 0.5:  # G listed: sorted positions, some past the end
                    kw["global_list"] = sorted(g.choice(maxk + 20, size=min(6, maxk + 20),
                                                        replace=False).tolist())
        if mask == MASK_PREFIX_LM:
            kw["prefix_len"] = int(rng.integers(0, maxk + 1))
        if mask in (MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE):
            nseg = int(rng.integers(1, 5))
            lo = int(rng.integers(0, max(1, maxk // 3)))
            cuts = sorted(rng.choice(np.arange(lo + 1, max(lo + 2, maxk)), size=nseg - 1,
                                     replace=False).tolist()) if nseg > 1 else []
            kw["segments"] = [lo] + [int(c) for c in cuts]
            if mask == MASK_CAUSAL_BLOCKWISE:
                kw["query_start"] = int(rng.integers(0, maxk + 1))
        norm = str(rng.choice(["softmax"] * 6 + ["relu", "sigmoid"]))
        dtype = "fp32" if rng.random() < 0.15 else "bf16"
        case = dict(name=f"u{seed}_{i:02d}_{shape}_{'varlen' if varlen else 'fixed'}_"
                         f"{MASK_NAMES[mask]}_{norm}_{dtype}",
                    shape=shape, lens=lens, varlen=varlen, mask=mask, norm=norm, dtype=dtype,
                    D=int(rng.choice([64, 128])), group=int(rng.choice([1, 2, 4, 8])),
                    hkv=int(rng.integers(1, 3)), alibi=bool(rng.random() < 0.3),
                    relpos=bool(rng.random() < 0.2),
                    softcap=float(rng.choice([0.0] * 4 + [20.0, 50.0, 400.0])),
                    seed=int(rng.integers(0, 1 << 30)), **kw)
        cases.append(case)
    return cases


CASES = _draw()


def _token_ids(starts, n):
    ids = [-1] * n
    for k, st in enumerate(starts):
        for pos in range(st, n):
            ids[pos] = k
    return ids


@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_unequal_lengths_random(c):
    log(f"[parity unequal random] {c['name']} (lq, lk) = {c['lens']} D={c['D']} "
        f"group={c['group']} hkv={c['hkv']} alibi={c['alibi']} relpos={c['relpos']} "
        f"softcap={c['softcap']}")
    g = torch.Generator().manual_seed(c["seed"])
    tdt = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
    hkv, D = c["hkv"], c["D"]
    hq = hkv * c["group"]
    sigma = 1.5 if (c["alibi"] or c["softcap"]) else 1.0
    lq = [a for a, _ in c["lens"]]
    lk = [b for _, b in c["lens"]]
    if c["varlen"]:
        qs, ks = (sum(lq), hq, D), (sum(lk), hkv, D)
    else:
        qs, ks = (len(lq), hq, lq[0], D), (len(lk), hkv, lk[0], D)
    q = (torch.randn(qs, generator=g) * sigma).to(tdt)
    k = (torch.randn(ks, generator=g) * sigma).to(tdt)
    v = torch.randn(ks, generator=g).to(tdt)
    slopes = alibi_slopes(hq) if c["alibi"] else None
    dev = "cuda:0"
    gkw, okw = {}, {}
    maxk = max(lk) if lk else 0
    if c["varlen"]:
        cuq = torch.tensor([0] + list(np.cumsum(lq)), dtype=torch.int32)
        cuk = torch.tensor([0] + list(np.cumsum(lk)), dtype=torch.int32)
        gkw.update(cu_seqlens_q=cuq.to(dev), cu_seqlens_k=cuk.to(dev), max_seqlen_q=max(lq),
                   max_seqlen_k=max(lk))
        okw.update(cu_seqlens_q=cuq, cu_seqlens_k=cuk)
    wl_, wr_ = c.get("window", (-1, -1))
    if "window" in c:
        gkw["window"] = c["window"]
    if "segments" in c:
        gkw["segment_starts"] = torch.tensor(c["segments"], dtype=torch.int32, device=dev)
        okw["token_ids"] = _token_ids(c["segments"], max(maxk, 1))
    if c["mask"] == MASK_GLOBAL_WINDOW and "global_list" in c:
        gkw["global_tokens"] = torch.tensor(c["global_list"], dtype=torch.int32, device=dev)
        okw["global_tokens"] = list(c["global_list"])
    elif c["mask"] == MASK_GLOBAL_WINDOW:
        gkw["num_global"] = c["num_global"]
        okw["global_tokens"] = list(range(c["num_global"]))
    o, lse = None, None
    res = fwd(q.to(dev), k.to(dev), v.to(dev), mask=MASK_NAMES[c["mask"]],
              alibi_slopes=slopes.to(dev) if slopes is not None else None, softcap=c["softcap"],
              relative_position=c["relpos"], norm=c["norm"], prefix_len=c.get("prefix_len", 0),
              query_start=c.get("query_start", 0), validate=True, **gkw)
    torch.cuda.synchronize()
    o, lse = res if isinstance(res, tuple) else (res, None)
    o_ref, lse_ref = oracle.attention(
        q, k, v, scale=D ** -0.5, mask=c["mask"], window_left=wl_, window_right=wr_,
        slopes=slopes, softcap=c["softcap"], prefix_len=c.get("prefix_len", 0),
        relpos=c["relpos"], norm={"softmax": 0, "relu": 1, "sigmoid": 2}[c["norm"]],
        query_start=c.get("query_start", 0), **okw)
    og = o.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(og).all()
    o_err = float(np.abs(og - o_ref).max()) if og.size else 0.0
    tol = O_TOL[c["dtype"]]
    if c["norm"] != "softmax":
        tol *= float(np.abs(o_ref).max()) if o_ref.size else 0.0
        log(f"  max|dO| = {o_err:.3e} (tol {tol:.2e})")
        assert o_err <= tol
        return
    lg = lse.cpu().numpy().astype(np.float64)
    inf_ref = np.isinf(lse_ref)
    assert np.array_equal(np.isinf(lg), inf_ref), "LSE -inf pattern differs"
    fin = ~inf_ref
    l_err = float(np.abs(lg[fin] - lse_ref[fin]).max()) if fin.any() else 0.0
    log(f"  max|dO| = {o_err:.3e} (tol {tol:.0e}), max|dLSE| = {l_err:.3e}")
    assert o_err <= tol
    assert l_err <= LSE_TOL

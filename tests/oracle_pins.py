"""Pins that tie the CPU oracle to facts fixed by the paper and by mathematics.

Each pin is a function `pin_x(lib)` that raises AssertionError when the oracle
loaded as `lib` disagrees with a fact that does not come from the oracle:
hand-derived closed forms (tests/golden/hand_cases.yaml), closed forms for
zero queries, reductions between variants, probability invariants, and the
fp64 library routine torch.nn.functional.scaled_dot_product_attention.

The same pins run against deliberately broken copies of the oracle
(test_oracle_mutants.py) to show that a plausible mistake fails at least one.
"""
from __future__ import annotations

import math
import os

import numpy as np
import torch
import torch.nn.functional as F
import yaml

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.yaml")
_NS = {"ln": math.log, "exp": math.exp, "e": math.e, "inf": math.inf, "sqrt": math.sqrt}
_MASKS = {"none": oracle.MASK_NONE, "causal": oracle.MASK_CAUSAL,
          "window": oracle.MASK_SLIDING_WINDOW, "prefix_lm": oracle.MASK_PREFIX_LM,
          "global_window": oracle.MASK_GLOBAL_WINDOW,
          "share_question": oracle.MASK_SHARE_QUESTION,
          "causal_blockwise": oracle.MASK_CAUSAL_BLOCKWISE}
_NORMS = {"softmax": oracle.NORM_SOFTMAX, "relu": oracle.NORM_RELU,
          "sigmoid": oracle.NORM_SIGMOID}


def _val(x):
    if isinstance(x, list):
        return [_val(y) for y in x]
    if isinstance(x, (int, float)):
        return float(x)
    return float(eval(str(x), {"__builtins__": {}}, _NS))  # fixture arithmetic only


def _close(a, b, tol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    inf_a, inf_b = np.isinf(a), np.isinf(b)
    assert np.array_equal(inf_a, inf_b) and np.array_equal(a[inf_a], b[inf_b]), \
        f"{what}: infinities differ\n{a}\n{b}"
    fin = ~inf_a
    err = np.max(np.abs(a[fin] - b[fin])) if fin.any() else 0.0
    assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.1e}\n{a}\n{b}"


def load_hand_cases():
    with open(GOLDEN) as f:
        return yaml.safe_load(f)["cases"]


def _run_case(lib, c):
    q = np.array(_val(c["q"]), dtype=np.float32)
    k = np.array(_val(c["k"]), dtype=np.float32)
    v = np.array(_val(c["v"]), dtype=np.float32)
    kw = dict(scale=_val(c["scale"]), mask=_MASKS[c["mask"]],
              window_left=int(c.get("window_left", -1)),
              window_right=int(c.get("window_right", -1)),
              softcap=_val(c.get("softcap", 0)), lib=lib,
              norm=_NORMS[c.get("norm", "softmax")], prefix_len=int(c.get("prefix_len", 0)),
              relpos=bool(c.get("relpos", 0)), query_start=int(c.get("query_start", 0)))
    if "token_ids" in c:
        kw["token_ids"] = np.array(c["token_ids"], dtype=np.int32)
    if "global_tokens" in c:
        kw["global_tokens"] = np.array(c["global_tokens"], dtype=np.int32)
    if "slopes" in c:
        kw["slopes"] = np.array(_val(c["slopes"]), dtype=np.float32)
    if "cu" in c:
        cu = np.array(c["cu"], dtype=np.int32)
        o, lse = oracle.attention(q[:, None, :], k[:, None, :], v[:, None, :],
                                  cu_seqlens_q=cu, cu_seqlens_k=cu, **kw)
        return o[:, 0, :], lse[0]
    if "heads" in c:
        o, lse = oracle.attention(q[None], k[None], v[None], **kw)
        return o[0], lse[0]
    o, lse = oracle.attention(q[None, None], k[None, None], v[None, None], **kw)
    return o[0, 0], lse[0, 0]


def pin_hand_cases(lib):
    """Every hand-derived case (inputs are fp32, so allow fp32 input rounding)."""
    for c in load_hand_cases():
        o, lse = _run_case(lib, c)
        _close(o, _val(c["o"]), 2e-6, c["name"] + " O")
        if "lse" in c:
            _close(lse, _val(c["lse"]), 2e-6, c["name"] + " LSE")
        else:  # ReLU / Sigmoid define no normaliser
            assert np.isnan(np.asarray(lse)).all(), c["name"] + ": LSE must be NaN"


def _rand(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(shape, generator=g, dtype=torch.float32) * scale)


def pin_probability_rows(lib):
    """Rows of P sum to one and P = exp(score - LSE) is consistent with O = P V."""
    B, H, S, D = 2, 3, 9, 5
    q, k, v = _rand((B, H, S, D), 1), _rand((B, H, S, D), 2), _rand((B, H, S, D), 3)
    slopes = torch.tensor([0.5, 0.25, 0.125])
    for kw in (dict(mask=oracle.MASK_NONE), dict(mask=oracle.MASK_CAUSAL),
               dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=2, window_right=1),
               dict(mask=oracle.MASK_NONE, softcap=1.5, slopes=slopes)):
        o, lse, p = oracle.attention(q, k, v, scale=0.4, want_probs=True, lib=lib, **kw)
        _close(p.sum(-1), np.ones((B, H, S)), 1e-12, f"row sums {kw}")
        assert (p >= 0).all()
        _close(o, np.einsum("bhij,bhjd->bhid", p, v.double().numpy()), 1e-12, f"O = P V {kw}")


def pin_constant_v(lib):
    """Constant V = c gives O = c whatever the scores."""
    B, H, S, D = 1, 2, 7, 4
    q, k = _rand((B, H, S, D), 4, 2.0), _rand((B, H, S, D), 5, 2.0)
    v = torch.full((B, H, S, D), -1.75)
    for kw in (dict(mask=oracle.MASK_NONE, softcap=3.0),
               dict(mask=oracle.MASK_CAUSAL, slopes=torch.tensor([0.3, 1.1])),
               dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=1, window_right=0)):
        o, _ = oracle.attention(q, k, v, scale=0.7, lib=lib, **kw)
        _close(o, np.full((B, H, S, D), -1.75), 1e-12, f"constant V {kw}")


def pin_causal_row0(lib):
    """Causal row 0 sees only key 0: O_0 = V_0, LSE_0 = scale * q_0 . k_0."""
    B, H, S, D = 2, 2, 6, 8
    q, k, v = _rand((B, H, S, D), 6), _rand((B, H, S, D), 7), _rand((B, H, S, D), 8)
    o, lse = oracle.attention(q, k, v, scale=0.3, mask=oracle.MASK_CAUSAL, lib=lib)
    _close(o[:, :, 0], v[:, :, 0].double().numpy(), 1e-12, "causal O_0")
    s00 = 0.3 * (q[:, :, 0].double() * k[:, :, 0].double()).sum(-1)
    _close(lse[:, :, 0], s00.numpy(), 1e-12, "causal LSE_0")


def pin_single_key_window(lib):
    """window_left = window_right = 0: each row sees only its own key."""
    B, H, S, D = 1, 2, 5, 3
    q, k, v = _rand((B, H, S, D), 9), _rand((B, H, S, D), 10), _rand((B, H, S, D), 11)
    o, lse = oracle.attention(q, k, v, scale=1.3, mask=oracle.MASK_SLIDING_WINDOW,
                              window_left=0, window_right=0, lib=lib)
    _close(o, v.double().numpy(), 1e-12, "window 0 O")
    _close(lse, (1.3 * (q.double() * k.double()).sum(-1)).numpy(), 1e-12, "window 0 LSE")


def pin_zero_query_counts(lib):
    """Q = 0: O_i = mean of visible V rows, LSE_i = ln(n_i), n_i from the mask."""
    S, D = 11, 3
    v = _rand((1, 1, S, D), 12)
    q = torch.zeros((1, 1, S, D))
    k = _rand((1, 1, S, D), 13)
    vn = v[0, 0].double().numpy()
    cases = [
        (dict(mask=oracle.MASK_NONE), lambda i: (0, S - 1)),
        (dict(mask=oracle.MASK_CAUSAL), lambda i: (0, i)),
        (dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=3, window_right=0),
         lambda i: (max(0, i - 3), i)),
        (dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=2, window_right=4),
         lambda i: (max(0, i - 2), min(S - 1, i + 4))),
        (dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=-1, window_right=2),
         lambda i: (0, min(S - 1, i + 2))),
    ]
    for kw, rng in cases:
        o, lse = oracle.attention(q, k, v, scale=1.0, lib=lib, **kw)
        for i in range(S):
            a, b = rng(i)
            _close(o[0, 0, i], vn[a:b + 1].mean(0), 1e-12, f"Q=0 O row {i} {kw}")
            _close(lse[0, 0, i], math.log(b - a + 1), 1e-12, f"Q=0 LSE row {i} {kw}")
    # bottom-right causal with Sq < Sk: query i sits at key position i + Sk - Sq
    sq = 4
    o, lse = oracle.attention(q[:, :, :sq], k, v, scale=1.0, mask=oracle.MASK_CAUSAL, lib=lib)
    for i in range(sq):
        n = i + S - sq + 1
        _close(o[0, 0, i], vn[:n].mean(0), 1e-12, f"bottom-right O row {i}")
        _close(lse[0, 0, i], math.log(n), 1e-12, f"bottom-right LSE row {i}")


def pin_zero_query_alibi(lib):
    """Q = 0 with ALiBi: weights r^|i-j| (r = e^-m), a two-sided geometric sum.

    With V = identity (D = S), O_i[j] = r^|i-j| / Z_i and
    Z_i = (1 - r^(i+1))/(1 - r) + r (1 - r^(S-1-i))/(1 - r)."""
    S = 9
    m = 0.37
    r = math.exp(-m)
    q = torch.zeros((1, 1, S, S))
    k = _rand((1, 1, S, S), 14)
    v = torch.eye(S).reshape(1, 1, S, S)
    o, lse = oracle.attention(q, k, v, scale=1.0, slopes=torch.tensor([m]), lib=lib)
    for i in range(S):
        z = (1 - r ** (i + 1)) / (1 - r) + r * (1 - r ** (S - 1 - i)) / (1 - r)
        _close(lse[0, 0, i], math.log(z), 1e-6, f"ALiBi Z row {i}")
        _close(o[0, 0, i], [r ** abs(i - j) / z for j in range(S)], 1e-6, f"ALiBi O row {i}")
    # causal: only j <= i, Z_i = (1 - r^(i+1)) / (1 - r)
    o, lse = oracle.attention(q, k, v, scale=1.0, mask=oracle.MASK_CAUSAL,
                              slopes=torch.tensor([m]), lib=lib)
    for i in range(S):
        z = (1 - r ** (i + 1)) / (1 - r)
        _close(lse[0, 0, i], math.log(z), 1e-6, f"causal ALiBi Z row {i}")


def pin_reductions(lib):
    """window >= Sk-1 is causal; C = 1e4 is (almost) no cap; zero slopes are no ALiBi."""
    B, H, S, D = 1, 2, 16, 8
    q, k, v = _rand((B, H, S, D), 15), _rand((B, H, S, D), 16), _rand((B, H, S, D), 17)
    oc, lc = oracle.attention(q, k, v, scale=0.35, mask=oracle.MASK_CAUSAL, lib=lib)
    for wl in (S - 1, S + 5, -1):
        ow, lw = oracle.attention(q, k, v, scale=0.35, mask=oracle.MASK_SLIDING_WINDOW,
                                  window_left=wl, window_right=0, lib=lib)
        _close(ow, oc, 0.0, f"window {wl} == causal O")
        _close(lw, lc, 0.0, f"window {wl} == causal LSE")
    op, lp = oracle.attention(q, k, v, scale=0.35, lib=lib)
    # |C tanh(s/C) - s| <= |s|^3 / (3 C^2); |s| < 5 here, so the gap is < 5e-7
    ocap, lcap = oracle.attention(q, k, v, scale=0.35, softcap=1e4, lib=lib)
    _close(ocap, op, 1e-6, "softcap 1e4 O")
    _close(lcap, lp, 1e-6, "softcap 1e4 LSE")
    oz, lz = oracle.attention(q, k, v, scale=0.35, slopes=torch.zeros(H), lib=lib)
    _close(oz, op, 0.0, "zero slopes O")
    _close(lz, lp, 0.0, "zero slopes LSE")


def pin_torch_sdpa(lib):
    """fp64 torch SDPA (library routine): plain, causal, GQA, window and ALiBi masks."""
    B, Hq, Hkv, S, D = 2, 4, 2, 13, 6
    q = _rand((B, Hq, S, D), 18, 1.5).double()
    k = _rand((B, Hkv, S, D), 19, 1.5).double()
    v = _rand((B, Hkv, S, D), 20).double()
    sc = 0.45
    # plain and causal with grouped-query heads (torch repeats kv heads in contiguous groups)
    for causal in (False, True):
        ref = F.scaled_dot_product_attention(q, k, v, is_causal=causal, scale=sc, enable_gqa=True)
        o, _ = oracle.attention(q, k, v, scale=sc, lib=lib,
                                mask=oracle.MASK_CAUSAL if causal else oracle.MASK_NONE)
        _close(o, ref.numpy(), 1e-12, f"sdpa causal={causal}")
    kr = k.repeat_interleave(Hq // Hkv, dim=1)
    vr = v.repeat_interleave(Hq // Hkv, dim=1)
    # band mask from torch's triangular routines: keys i-3 .. i+1 visible
    band = torch.ones(S, S, dtype=torch.bool).tril(1).triu(-3)
    ref = F.scaled_dot_product_attention(q, kr, vr, attn_mask=band, scale=sc)
    o, _ = oracle.attention(q, k, v, scale=sc, mask=oracle.MASK_SLIDING_WINDOW,
                            window_left=3, window_right=1, lib=lib)
    _close(o, ref.numpy(), 1e-12, "sdpa band")
    # ALiBi as an additive float mask: -slope_h * |i - j|
    slopes = torch.tensor([0.5, 0.25, 0.125, 0.0625], dtype=torch.float64)
    idx = torch.arange(S, dtype=torch.float64)
    dist = (idx[:, None] - idx[None, :]).abs()
    bias = -slopes[:, None, None] * dist[None]
    ref = F.scaled_dot_product_attention(q, kr, vr, attn_mask=bias[None], scale=sc)
    o, lse = oracle.attention(q, k, v, scale=sc, slopes=slopes.float(), lib=lib)
    _close(o, ref.numpy(), 1e-12, "sdpa alibi")
    # LSE against torch.logsumexp of the same biased scores
    s = sc * torch.einsum("bhid,bhjd->bhij", q, kr) + bias[None]
    _close(lse, torch.logsumexp(s, -1).numpy(), 1e-12, "logsumexp alibi")


def pin_gqa_equals_repeated(lib):
    """GQA equals MHA over K/V heads repeated in contiguous groups."""
    B, Hq, Hkv, S, D = 1, 6, 2, 10, 4
    q, k, v = _rand((B, Hq, S, D), 21), _rand((B, Hkv, S, D), 22), _rand((B, Hkv, S, D), 23)
    kw = dict(scale=0.5, mask=oracle.MASK_SLIDING_WINDOW, window_left=4, window_right=0,
              softcap=2.5, slopes=torch.linspace(0.1, 0.6, Hq), lib=lib)
    og, lg = oracle.attention(q, k, v, **kw)
    om, lm = oracle.attention(q, k.repeat_interleave(3, 1), v.repeat_interleave(3, 1), **kw)
    _close(og, om, 0.0, "GQA O")
    _close(lg, lm, 0.0, "GQA LSE")


def pin_varlen_concat(lib):
    """Varlen equals independent fixed-length runs per sequence (incl. empty ones)."""
    lens = [5, 0, 1, 9, 3]
    Hq, Hkv, D = 4, 2, 6
    T = sum(lens)
    q, k, v = _rand((T, Hq, D), 24), _rand((T, Hkv, D), 25), _rand((T, Hkv, D), 26)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    slopes = torch.tensor([0.2, 0.4, 0.6, 0.8])
    for kw in (dict(mask=oracle.MASK_CAUSAL),
               dict(mask=oracle.MASK_NONE, slopes=slopes, softcap=3.0),
               dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=2, window_right=0)):
        ov, lv = oracle.attention(q, k, v, scale=0.6, cu_seqlens_q=cu, cu_seqlens_k=cu,
                                  lib=lib, **kw)
        for s, n in enumerate(lens):
            if n == 0:
                continue
            a = cu[s]
            sl = slice(a, a + n)
            of, lf = oracle.attention(q[sl].permute(1, 0, 2)[None], k[sl].permute(1, 0, 2)[None],
                                      v[sl].permute(1, 0, 2)[None], scale=0.6, lib=lib, **kw)
            _close(ov[sl], of[0].transpose(1, 0, 2), 0.0, f"varlen O seq {s} {kw}")
            _close(lv[:, sl], lf[0], 0.0, f"varlen LSE seq {s} {kw}")


def pin_varlen_unequal_lengths(lib):
    """Varlen with separate query/key lengths, Q = 0: bottom-right causal per sequence.

    Query i of a sequence with Lq queries and Lk keys sees keys 0..i+Lk-Lq, so
    n_i = clip(i + Lk - Lq + 1, 0, Lk); O_i is the mean of those V rows and
    LSE_i = ln n_i (an empty row has O = 0, LSE = -inf)."""
    lq = [3, 4, 2, 0, 2]
    lk = [5, 2, 0, 3, 2]
    cuq = np.concatenate([[0], np.cumsum(lq)]).astype(np.int32)
    cuk = np.concatenate([[0], np.cumsum(lk)]).astype(np.int32)
    D = 2
    q = torch.zeros((sum(lq), 1, D))
    k = _rand((sum(lk), 1, D), 30)
    v = _rand((sum(lk), 1, D), 31)
    o, lse = oracle.attention(q, k, v, scale=1.0, mask=oracle.MASK_CAUSAL,
                              cu_seqlens_q=cuq, cu_seqlens_k=cuk, lib=lib)
    vn = v[:, 0].double().numpy()
    for s_, (a, b) in enumerate(zip(lq, lk)):
        for i in range(a):
            n = min(max(i + b - a + 1, 0), b)
            t = cuq[s_] + i
            if n == 0:
                _close(o[t, 0], np.zeros(D), 0.0, f"empty row seq {s_} i {i}")
                _close(lse[0, t], -math.inf, 0.0, f"empty LSE seq {s_} i {i}")
            else:
                _close(o[t, 0], vn[cuk[s_]:cuk[s_] + n].mean(0), 1e-12, f"O seq {s_} i {i}")
                _close(lse[0, t], math.log(n), 1e-12, f"LSE seq {s_} i {i}")


def pin_row_subset(lib):
    """Computing a subset of rows gives the same values as computing all rows."""
    B, H, S, D = 2, 3, 7, 4
    q, k, v = _rand((B, H, S, D), 27), _rand((B, H, S, D), 28), _rand((B, H, S, D), 29)
    o, lse = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_CAUSAL, lib=lib)
    rows = [0, 5, 17, 41]
    os_, ls = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_CAUSAL, rows=rows, lib=lib)
    flat_o, flat_os = o.reshape(-1, D), os_.reshape(-1, D)
    _close(flat_os[rows], flat_o[rows], 0.0, "row subset O")
    _close(ls.reshape(-1)[rows], lse.reshape(-1)[rows], 0.0, "row subset LSE")
    assert np.isnan(np.delete(ls.reshape(-1), rows)).all()


def _zero_q_counts(lib, S, visible_sets, what, sq=None, **kw):
    """Q = 0: O_i = mean of the visible V rows, LSE_i = ln n_i (O = 0, LSE = -inf
    for an empty row). visible_sets[i] is the set of keys row i must see; with
    sq < S there are sq queries against S keys."""
    D = 3
    sq = S if sq is None else sq
    v = _rand((1, 1, S, D), 40)
    q = torch.zeros((1, 1, sq, D))
    k = _rand((1, 1, S, D), 41)
    o, lse = oracle.attention(q, k, v, scale=1.0, lib=lib, **kw)
    vn = v[0, 0].double().numpy()
    for i in range(sq):
        js = sorted(visible_sets[i])
        if not js:
            _close(o[0, 0, i], np.zeros(D), 0.0, f"{what}: empty row {i} O")
            _close(lse[0, 0, i], -math.inf, 0.0, f"{what}: empty row {i} LSE")
            continue
        _close(o[0, 0, i], vn[js].mean(0), 1e-12, f"{what}: row {i} O")
        _close(lse[0, 0, i], math.log(len(js)), 1e-12, f"{what}: row {i} LSE")


def pin_prefix_lm(lib):
    """PrefixLM (Appendix A): keys j < L_p for every row, else j <= i; L_p = 0 and
    L_p = 1 reduce to causal, L_p >= S to no mask."""
    S = 13
    for lp in (0, 1, 4, 12, 13, 20):
        sets = [set(range(min(lp, S))) | set(range(i + 1)) for i in range(S)]
        _zero_q_counts(lib, S, sets, f"prefix {lp}", mask=oracle.MASK_PREFIX_LM, prefix_len=lp)
    B, H, D = 1, 2, 8
    q, k, v = _rand((B, H, S, D), 42), _rand((B, H, S, D), 43), _rand((B, H, S, D), 44)
    oc, lc = oracle.attention(q, k, v, scale=0.4, mask=oracle.MASK_CAUSAL, lib=lib)
    on, ln_ = oracle.attention(q, k, v, scale=0.4, lib=lib)
    for lp, (oe, le) in ((0, (oc, lc)), (1, (oc, lc)), (S, (on, ln_)), (S + 3, (on, ln_))):
        op, lp_ = oracle.attention(q, k, v, scale=0.4, mask=oracle.MASK_PREFIX_LM, prefix_len=lp,
                                   lib=lib)
        _close(op, oe, 0.0, f"prefix {lp} reduction O")
        _close(lp_, le, 0.0, f"prefix {lp} reduction LSE")


def pin_relative_position(lib):
    """Score = S + (i - j) (Appendix A). With Q = 0 and V = I the weights of row i
    are e^(i'-j) / Z_i, Z_i a geometric sum; i' = i + Sk - Sq."""
    S = 7
    q = torch.zeros((1, 1, S, S))
    k = _rand((1, 1, S, S), 45)
    v = torch.eye(S).reshape(1, 1, S, S)
    e = math.e
    o, lse = oracle.attention(q, k, v, scale=1.0, mask=oracle.MASK_CAUSAL, relpos=True, lib=lib)
    for i in range(S):
        z = (e ** (i + 1) - 1) / (e - 1)  # sum_{m=0..i} e^m
        _close(lse[0, 0, i], math.log(z), 1e-12, f"relpos causal Z row {i}")
        _close(o[0, 0, i], [e ** (i - j) / z if j <= i else 0.0 for j in range(S)], 1e-12,
               f"relpos causal O row {i}")
    o, lse = oracle.attention(q, k, v, scale=1.0, relpos=True, lib=lib)
    for i in range(S):
        z = sum(e ** (i - j) for j in range(S))
        _close(lse[0, 0, i], math.log(z), 1e-12, f"relpos Z row {i}")
    # the term is added after the soft-cap: with Q = 0 the capped score is
    # C tanh(0) = 0 for any C, so the weights stay e^(i-j) (capping the sum
    # would give e^(C tanh((i-j)/C)))
    for cap in (0.5, 2.0):
        o, lse = oracle.attention(q, k, v, scale=1.0, mask=oracle.MASK_CAUSAL, relpos=True,
                                  softcap=cap, lib=lib)
        for i in range(S):
            z = (e ** (i + 1) - 1) / (e - 1)
            _close(lse[0, 0, i], math.log(z), 1e-12, f"relpos after cap {cap} Z row {i}")
            _close(o[0, 0, i], [e ** (i - j) / z if j <= i else 0.0 for j in range(S)], 1e-12,
                   f"relpos after cap {cap} O row {i}")
    # bottom-right alignment: 3 queries against 7 keys, query i at position i + 4
    o, lse = oracle.attention(q[:, :, 4:], k, v, scale=1.0, mask=oracle.MASK_CAUSAL,
                              relpos=True, lib=lib)
    for i in range(3):
        ii = i + 4
        z = (e ** (ii + 1) - 1) / (e - 1)
        _close(lse[0, 0, i], math.log(z), 1e-12, f"relpos Sq<Sk Z row {i}")


def pin_relu_sigmoid(lib):
    """ReLU(S)/L and Sigmoid(S)/L (Appendix A): with Q = 0 every score is 0, so
    Sigmoid gives O_i = n_i * mean(V_visible) / (2 L) and ReLU gives O = 0; P rows
    equal act(S)/L exactly; masked keys get weight 0."""
    S, D = 9, 4
    v = _rand((1, 1, S, D), 46)
    k = _rand((1, 1, S, D), 47)
    q0 = torch.zeros((1, 1, S, D))
    vn = v[0, 0].double().numpy()
    o, lse = oracle.attention(q0, k, v, scale=1.0, mask=oracle.MASK_CAUSAL,
                              norm=oracle.NORM_SIGMOID, lib=lib)
    for i in range(S):
        _close(o[0, 0, i], vn[:i + 1].sum(0) / (2 * S), 1e-12, f"sigmoid Q=0 row {i}")
    assert np.isnan(lse).all()
    o, _ = oracle.attention(q0, k, v, scale=1.0, norm=oracle.NORM_RELU, lib=lib)
    _close(o, np.zeros_like(o), 0.0, "relu Q=0")
    # P = act(scale * q.k)/L on random scores, against scipy-free closed forms
    q = _rand((1, 1, S, D), 48, 1.5)
    s = 0.6 * torch.einsum("bhid,bhjd->bhij", q.double(), k.double()).numpy()
    for norm, act in ((oracle.NORM_RELU, lambda x: np.maximum(x, 0.0)),
                      (oracle.NORM_SIGMOID, lambda x: 1.0 / (1.0 + np.exp(-x)))):
        o, _, p = oracle.attention(q, k, v, scale=0.6, norm=norm, want_probs=True, lib=lib)
        _close(p, act(s) / S, 1e-12, f"norm {norm} P")
        o, _, p = oracle.attention(q, k, v, scale=0.6, norm=norm, mask=oracle.MASK_CAUSAL,
                                   want_probs=True, lib=lib)
        tri = np.tril(np.ones((S, S), dtype=bool))
        _close(p[0, 0][~tri], np.zeros((~tri).sum()), 0.0, f"norm {norm} masked P")
        _close(p[0, 0][tri], (act(s) / S)[0, 0][tri], 1e-12, f"norm {norm} causal P")


def pin_global_window(lib):
    """Global Sliding Window (Appendix A): |i-j| <= w, or i in G, or j in G.
    G empty reduces to the symmetric sliding window."""
    S = 14
    for w, G in ((0, [0]), (2, [0, 1]), (1, [5, 11]), (3, []), (0, list(range(S)))):
        sets = []
        for i in range(S):
            if i in G:
                sets.append(set(range(S)))
            else:
                sets.append({j for j in range(S) if abs(i - j) <= w} | set(G))
        _zero_q_counts(lib, S, sets, f"global w={w} G={G}", mask=oracle.MASK_GLOBAL_WINDOW,
                       window_left=w, window_right=w, global_tokens=G)
    B, H, D = 1, 2, 6
    q, k, v = _rand((B, H, S, D), 49), _rand((B, H, S, D), 50), _rand((B, H, S, D), 51)
    ow, lw = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_SLIDING_WINDOW,
                              window_left=3, window_right=3, lib=lib)
    og, lg = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_GLOBAL_WINDOW,
                              window_left=3, window_right=3, global_tokens=[], lib=lib)
    _close(og, ow, 0.0, "global G=[] O")
    _close(lg, lw, 0.0, "global G=[] LSE")


def _ids_from_starts(S, starts):
    ids = [-1] * S
    for k, st in enumerate(starts):
        for p in range(st, S):
            ids[p] = k
    return ids


def pin_share_question(lib):
    """Share Question (Appendix A): a prompt row sees the prompt causally; a row of
    response A_k sees the prompt and A_k up to itself. No responses is causal."""
    S = 15
    for starts in ([4, 7, 12], [0, 5], [3], [1, 2, 3, 4]):
        ids = _ids_from_starts(S, starts)
        sets = []
        for i in range(S):
            if ids[i] < 0:
                sets.append(set(range(i + 1)))
            else:
                a = starts[ids[i]]
                sets.append(set(range(starts[0])) | set(range(a, i + 1)))
        _zero_q_counts(lib, S, sets, f"share question {starts}", mask=oracle.MASK_SHARE_QUESTION,
                       token_ids=ids)
    B, H, D = 1, 2, 6
    q, k, v = _rand((B, H, S, D), 52), _rand((B, H, S, D), 53), _rand((B, H, S, D), 54)
    oc, lc = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_CAUSAL, lib=lib)
    os_, ls = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_SHARE_QUESTION,
                               token_ids=[-1] * S, lib=lib)
    _close(os_, oc, 0.0, "share question all-prompt O")
    _close(ls, lc, 0.0, "share question all-prompt LSE")


def pin_causal_blockwise(lib):
    """Causal Blockwise (Appendix A): rows before L_q see their own document up to
    themselves, test-query rows see every key up to themselves. L_q = 0 or a
    single document reduce to causal."""
    S = 16
    for starts, lq_ in (([0, 3, 8], 12), ([0, 5, 6, 10], 16), ([2, 9], 9), ([0, 4], 0)):
        ids = _ids_from_starts(S, starts)
        sets = []
        for i in range(S):
            if i >= lq_:
                sets.append(set(range(i + 1)))
            else:
                sets.append({j for j in range(i + 1) if ids[j] == ids[i]})
        _zero_q_counts(lib, S, sets, f"blockwise {starts} Lq={lq_}",
                       mask=oracle.MASK_CAUSAL_BLOCKWISE, token_ids=ids, query_start=lq_)
    B, H, D = 1, 2, 6
    q, k, v = _rand((B, H, S, D), 55), _rand((B, H, S, D), 56), _rand((B, H, S, D), 57)
    oc, lc = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_CAUSAL, lib=lib)
    for ids, lq_ in (([0] * S, S), (_ids_from_starts(S, [0, 7]), 0)):
        ob, lb = oracle.attention(q, k, v, scale=0.5, mask=oracle.MASK_CAUSAL_BLOCKWISE,
                                  token_ids=ids, query_start=lq_, lib=lib)
        _close(ob, oc, 0.0, f"blockwise reduction O (Lq={lq_})")
        _close(lb, lc, 0.0, f"blockwise reduction LSE (Lq={lq_})")


def _visible_sets(kind, sq, sk, *, wl=-1, wr=-1, lp=0, G=(), ids=None, lq_=0):
    """Keys visible to each of sq queries against sk keys, written from the
    paper's case analyses at the key-axis position i' = i + sk - sq."""
    sets = []
    for i in range(sq):
        ii = i + sk - sq
        keys = range(sk)
        if kind == oracle.MASK_NONE:
            vis = set(keys)
        elif kind == oracle.MASK_CAUSAL:
            vis = {j for j in keys if j <= ii}
        elif kind == oracle.MASK_SLIDING_WINDOW:
            vis = {j for j in keys if (wl < 0 or ii - j <= wl) and (wr < 0 or j - ii <= wr)}
        elif kind == oracle.MASK_PREFIX_LM:
            vis = {j for j in keys if j < lp or j <= ii}
        elif kind == oracle.MASK_GLOBAL_WINDOW:
            vis = set(keys) if ii in G else \
                {j for j in keys if abs(ii - j) <= wl or j in G}
        elif kind == oracle.MASK_SHARE_QUESTION:
            vis = set() if ii < 0 else {j for j in keys if j <= ii and (
                (ids[ii] < 0 and ids[j] < 0) or (ids[ii] >= 0 and ids[j] in (-1, ids[ii])))}
        elif kind == oracle.MASK_CAUSAL_BLOCKWISE:
            vis = set() if ii < 0 else {j for j in keys if j <= ii and (
                ii >= lq_ or ids[ii] == ids[j])}
        else:
            raise ValueError(kind)
        sets.append(vis)
    return sets


def pin_bottom_right_counts(lib):
    """Q = 0 with fewer (and more) queries than keys: every mask kind places
    query i at key position i' = i + Sk - Sq (O = mean of the visible V rows,
    LSE = ln n_i; rows with no visible key give O = 0, LSE = -inf)."""
    S = 13
    ids_sq = _ids_from_starts(S, [4, 7, 11])
    ids_bw = _ids_from_starts(S, [0, 3, 8])
    cases = [
        (dict(mask=oracle.MASK_CAUSAL), dict()),
        (dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=2, window_right=0), dict(wl=2, wr=0)),
        (dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=1, window_right=3), dict(wl=1, wr=3)),
        (dict(mask=oracle.MASK_PREFIX_LM, prefix_len=3), dict(lp=3)),
        (dict(mask=oracle.MASK_GLOBAL_WINDOW, window_left=1, window_right=1,
              global_tokens=[2, 9]), dict(wl=1, G=(2, 9))),
        (dict(mask=oracle.MASK_SHARE_QUESTION, token_ids=ids_sq), dict(ids=ids_sq)),
        (dict(mask=oracle.MASK_CAUSAL_BLOCKWISE, token_ids=ids_bw, query_start=10),
         dict(ids=ids_bw, lq_=10)),
    ]
    for kw, skw in cases:
        for sq in (1, 5, S):
            sets = _visible_sets(kw["mask"], sq, S, **skw)
            _zero_q_counts(lib, S, sets, f"Sq={sq} Sk={S} {kw}", sq=sq, **kw)
    # more queries than keys: the first Sq - Sk rows of a causal mask see nothing
    for kw, skw in cases[:4]:
        sk = 6
        sets = _visible_sets(kw["mask"], 9, sk, **skw)
        D = 3
        v = _rand((1, 1, sk, D), 60)
        o, lse = oracle.attention(torch.zeros((1, 1, 9, D)), _rand((1, 1, sk, D), 61), v,
                                  scale=1.0, lib=lib, **kw)
        vn = v[0, 0].double().numpy()
        for i, vis in enumerate(sets):
            js = sorted(vis)
            if not js:
                _close(o[0, 0, i], np.zeros(D), 0.0, f"Sq>Sk empty row {i} {kw}")
                _close(lse[0, 0, i], -math.inf, 0.0, f"Sq>Sk empty LSE {i} {kw}")
            else:
                _close(o[0, 0, i], vn[js].mean(0), 1e-12, f"Sq>Sk row {i} {kw}")
                _close(lse[0, 0, i], math.log(len(js)), 1e-12, f"Sq>Sk LSE {i} {kw}")


def pin_alibi_bottom_right(lib):
    """Q = 0, ALiBi, Sq < Sk: query i at position i' = i + Sk - Sq weighs key j by
    r^|i' - j| (r = e^-m); with V = identity O_i[j] = r^|i'-j| / Z_i, Z_i a
    two-sided geometric sum (non-causal) or one-sided (causal)."""
    S, sq, m = 9, 4, 0.37
    r = math.exp(-m)
    q = torch.zeros((1, 1, sq, S))
    k = _rand((1, 1, S, S), 62)
    v = torch.eye(S).reshape(1, 1, S, S)
    o, lse = oracle.attention(q, k, v, scale=1.0, slopes=torch.tensor([m]), lib=lib)
    oc, lc = oracle.attention(q, k, v, scale=1.0, slopes=torch.tensor([m]),
                              mask=oracle.MASK_CAUSAL, lib=lib)
    for i in range(sq):
        ii = i + S - sq
        z = (1 - r ** (ii + 1)) / (1 - r) + r * (1 - r ** (S - 1 - ii)) / (1 - r)
        _close(lse[0, 0, i], math.log(z), 1e-6, f"ALiBi Sq<Sk Z row {i}")
        _close(o[0, 0, i], [r ** abs(ii - j) / z for j in range(S)], 1e-6,
               f"ALiBi Sq<Sk O row {i}")
        zc = (1 - r ** (ii + 1)) / (1 - r)
        _close(lc[0, 0, i], math.log(zc), 1e-6, f"causal ALiBi Sq<Sk Z row {i}")
        _close(oc[0, 0, i], [r ** (ii - j) / zc if j <= ii else 0.0 for j in range(S)], 1e-6,
               f"causal ALiBi Sq<Sk O row {i}")


def pin_norm_key_length(lib):
    """ReLU / Sigmoid divide by L = the key length of the row's sequence, also
    when it differs from the query length: with Q = 0, Sigmoid gives
    O_i = sum of the visible V rows / (2 Lk)."""
    D = 3
    for sq, sk, mask in ((2, 7, oracle.MASK_NONE), (3, 7, oracle.MASK_CAUSAL),
                         (8, 5, oracle.MASK_CAUSAL)):
        v = _rand((1, 1, sk, D), 63)
        o, lse = oracle.attention(torch.zeros((1, 1, sq, D)), _rand((1, 1, sk, D), 64), v,
                                  scale=1.0, mask=mask, norm=oracle.NORM_SIGMOID, lib=lib)
        vn = v[0, 0].double().numpy()
        for i, vis in enumerate(_visible_sets(mask, sq, sk)):
            js = sorted(vis)
            want = vn[js].sum(0) / (2 * sk) if js else np.zeros(D)
            _close(o[0, 0, i], want, 1e-12, f"sigmoid L=Lk sq={sq} sk={sk} row {i}")
        assert np.isnan(lse).all()
    # packed sequences with their own query and key lengths
    lq, lk = [2, 5, 1], [6, 3, 4]
    cuq = np.concatenate([[0], np.cumsum(lq)]).astype(np.int32)
    cuk = np.concatenate([[0], np.cumsum(lk)]).astype(np.int32)
    v = _rand((sum(lk), 1, D), 65)
    o, _ = oracle.attention(torch.zeros((sum(lq), 1, D)), _rand((sum(lk), 1, D), 66), v,
                            scale=1.0, mask=oracle.MASK_CAUSAL, norm=oracle.NORM_SIGMOID,
                            cu_seqlens_q=cuq, cu_seqlens_k=cuk, lib=lib)
    vn = v[:, 0].double().numpy()
    for s_, (a, b) in enumerate(zip(lq, lk)):
        for i, vis in enumerate(_visible_sets(oracle.MASK_CAUSAL, a, b)):
            js = [cuk[s_] + j for j in sorted(vis)]
            want = vn[js].sum(0) / (2 * b) if js else np.zeros(D)
            _close(o[cuq[s_] + i, 0], want, 1e-12, f"varlen sigmoid L=Lk seq {s_} row {i}")


_REDUCTION_VARIANTS = [
    dict(mask=oracle.MASK_NONE),
    dict(mask=oracle.MASK_CAUSAL),
    dict(mask=oracle.MASK_SLIDING_WINDOW, window_left=3, window_right=1),
    dict(mask=oracle.MASK_PREFIX_LM, prefix_len=4),
    dict(mask=oracle.MASK_GLOBAL_WINDOW, window_left=2, window_right=2, global_tokens=[2, 8]),
    dict(mask=oracle.MASK_SHARE_QUESTION, token_ids=_ids_from_starts(12, [3, 6, 10])),
    dict(mask=oracle.MASK_CAUSAL_BLOCKWISE, token_ids=_ids_from_starts(12, [0, 4, 7]),
         query_start=9),
]
_REDUCTION_MODS = [
    dict(),
    dict(slopes=[0.3, 0.7, 0.2, 0.9]),
    dict(relpos=True),
    dict(softcap=1.5, relpos=True, slopes=[0.5, 0.1, 0.25, 0.05]),
    dict(norm=oracle.NORM_RELU, slopes=[0.3, 0.7, 0.2, 0.9]),
    dict(norm=oracle.NORM_SIGMOID, relpos=True, softcap=2.0),
]


def pin_shape_reduction(lib):
    """Fewer queries than keys is the tail of the square problem: the Sq rows of
    an Sq x Sk run equal the last Sq rows of the Sk x Sk run on the same keys,
    for every mask kind, bias, soft-cap and normalisation (fixed length and
    packed sequences). This is what placing query i at key position
    i + Sk - Sq means; it fixes that alignment, and L = Lk for ReLU / Sigmoid,
    in every variant at once."""
    Sk, Hq, Hkv, D = 12, 4, 2, 5
    q = _rand((1, Hq, Sk, D), 70, 1.3)
    k = _rand((1, Hkv, Sk, D), 71, 1.3)
    v = _rand((1, Hkv, Sk, D), 72)
    for vk in _REDUCTION_VARIANTS:
        for mk in _REDUCTION_MODS:
            kw = dict(vk, **mk)
            if "slopes" in kw:
                kw["slopes"] = torch.tensor(kw["slopes"])
            of, lf = oracle.attention(q, k, v, scale=0.45, lib=lib, **kw)
            for sq in (1, 5):
                os_, ls = oracle.attention(q[:, :, Sk - sq:], k, v, scale=0.45, lib=lib, **kw)
                _close(os_, of[:, :, Sk - sq:], 0.0, f"Sq={sq} tail O {kw}")
                if kw.get("norm", oracle.NORM_SOFTMAX) == oracle.NORM_SOFTMAX:
                    _close(ls, lf[:, :, Sk - sq:], 0.0, f"Sq={sq} tail LSE {kw}")
    # packed: every sequence keeps its last lq_s queries of lk_s
    lk = [12, 7, 1, 9]
    lq = [5, 7, 0, 2]
    T = sum(lk)
    qp = _rand((T, Hq, D), 73, 1.3)
    kp = _rand((T, Hkv, D), 74, 1.3)
    vp = _rand((T, Hkv, D), 75)
    cuk = np.concatenate([[0], np.cumsum(lk)]).astype(np.int32)
    cuq = np.concatenate([[0], np.cumsum(lq)]).astype(np.int32)
    tail = np.concatenate([np.arange(cuk[s + 1] - lq[s], cuk[s + 1]) for s in range(len(lk))])
    for vk in _REDUCTION_VARIANTS:
        for mk in _REDUCTION_MODS:
            kw = dict(vk, **mk)
            if "slopes" in kw:
                kw["slopes"] = torch.tensor(kw["slopes"])
            of, lf = oracle.attention(qp, kp, vp, scale=0.45, cu_seqlens_q=cuk, cu_seqlens_k=cuk,
                                      lib=lib, **kw)
            os_, ls = oracle.attention(qp[torch.as_tensor(tail)], kp, vp, scale=0.45,
                                       cu_seqlens_q=cuq, cu_seqlens_k=cuk, lib=lib, **kw)
            _close(os_, of[tail], 0.0, f"varlen tail O {kw}")
            if kw.get("norm", oracle.NORM_SOFTMAX) == oracle.NORM_SOFTMAX:
                _close(ls, lf[:, tail], 0.0, f"varlen tail LSE {kw}")


ALL_PINS = [pin_hand_cases, pin_probability_rows, pin_constant_v, pin_causal_row0,
            pin_single_key_window, pin_zero_query_counts, pin_zero_query_alibi,
            pin_reductions, pin_torch_sdpa, pin_gqa_equals_repeated, pin_varlen_concat,
            pin_varlen_unequal_lengths, pin_row_subset, pin_prefix_lm, pin_relative_position,
            pin_relu_sigmoid, pin_global_window, pin_share_question, pin_causal_blockwise,
            pin_bottom_right_counts, pin_alibi_bottom_right, pin_norm_key_length,
            pin_shape_reduction]


def failing_pins(lib):
    """Names of the pins that fail for `lib` (empty when all hold)."""
    bad = []
    for pin in ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError) as e:  # noqa: PERF203
            bad.append((pin.__name__, str(e).splitlines()[0] if str(e) else ""))
    return bad

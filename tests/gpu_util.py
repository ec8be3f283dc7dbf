"""Helpers shared by the GPU tests: run the HIP path through the C ABI on
seeded inputs and compare with the CPU oracle element by element."""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
import paper_2605_05023_amd as attn
from paper_2605_05023_amd.workloads import Inputs

# Tolerances on the output O (max abs error) by dtype, and on LSE.
O_TOL = {"bf16": 2e-2, "fp32": 1e-4}
LSE_TOL = 1e-3
# ReLU / Sigmoid outputs are sums scaled by 1/L, of order 1/sqrt(L), so an
# absolute bar would not test them: their error must stay within the same
# fraction of the output's own scale, max|dO| <= O_TOL * max|O_ref|. The
# arithmetic allows it: P is rounded to bf16 (relative 2^-8 at most) and O to its dtype.


def gpu_available() -> bool:
    return torch.cuda.is_available()


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(inp: Inputs, *, out=None, lse=None, q=None, k=None, v=None, **extra):
    """Run the library on `inp` (tensors moved to cuda:0 unless given); `extra`
    passes further fwd arguments (schedule overrides, validate). Returns
    (out, lse); lse is None for the ReLU / Sigmoid normalisations."""
    dev = torch.device("cuda:0")
    q = inp.q.to(dev) if q is None else q
    k = inp.k.to(dev) if k is None else k
    v = inp.v.to(dev) if v is None else v
    res = attn.fwd(q, k, v, out=out, lse=lse, **inp.variant_kwargs(dev), **extra)
    return res if isinstance(res, tuple) else (res, None)


def rows_to_index(inp: Inputs, rows):
    """Flat LSE row ids -> index tuples into O."""
    rows = np.asarray(rows, dtype=np.int64)
    if inp.cu_seqlens is not None:
        T = inp.total_tokens
        return rows % T, rows // T          # (token, head)
    B, H, S, _ = inp.q.shape
    return rows // (H * S), (rows // S) % H, rows % S


def compare(inp: Inputs, o_gpu, lse_gpu, rows=None, *, o_tol=None, lse_tol=LSE_TOL, ref=None):
    """Max abs errors of O and LSE against the oracle on `rows` (all rows if None)."""
    o_ref, lse_ref = ref if ref is not None else oracle.attention_inputs(inp, rows=rows)
    o_tol = O_TOL[inp.wl.dtype] if o_tol is None else o_tol
    softmax = inp.wl.norm == "softmax"
    if rows is None:
        og = o_gpu.float().cpu().numpy().astype(np.float64)
        lg = lse_gpu.cpu().numpy().astype(np.float64) if softmax else None
        orf, lrf = o_ref, lse_ref
    else:
        idx = rows_to_index(inp, rows)
        tidx = tuple(torch.as_tensor(i, device=o_gpu.device) for i in idx)
        og = o_gpu[tidx].float().cpu().numpy().astype(np.float64)
        lg = None
        if softmax:
            lg = lse_gpu.reshape(-1)[torch.as_tensor(rows, device=lse_gpu.device)].cpu().numpy()
            lg = lg.astype(np.float64)
        orf = o_ref[idx]
        lrf = lse_ref.reshape(-1)[rows]
    assert np.isfinite(og).all(), "non-finite values in O"
    o_err = float(np.max(np.abs(og - orf))) if og.size else 0.0
    if not softmax:  # no LSE; O bar relative to the output's scale
        scale = float(np.max(np.abs(orf))) if orf.size else 0.0
        return o_err, 0.0, o_tol * scale, lse_tol
    inf_ref = np.isinf(lrf)
    assert np.array_equal(np.isinf(lg), inf_ref), "LSE -inf pattern differs"
    assert (lg[inf_ref] == lrf[inf_ref]).all()
    fin = ~inf_ref
    lse_err = float(np.max(np.abs(lg[fin] - lrf[fin]))) if fin.any() else 0.0
    return o_err, lse_err, o_tol, lse_tol


def assert_parity(inp, o_gpu, lse_gpu, rows=None, label="", **kw):
    o_err, lse_err, o_tol, lse_tol = compare(inp, o_gpu, lse_gpu, rows, **kw)
    log(f"  {label}: max|dO| = {o_err:.3e} (tol {o_tol:.0e}), max|dLSE| = {lse_err:.3e} "
        f"(tol {lse_tol:.0e})")
    assert o_err <= o_tol, f"{label}: O error {o_err} > {o_tol}"
    assert lse_err <= lse_tol, f"{label}: LSE error {lse_err} > {lse_tol}"
    return o_err, lse_err


def sample_rows(inp: Inputs, n_random: int, seed: int = 0, block_m: int = 128):
    """Flat LSE row ids: n_random seeded random rows plus structural ones (first
    and last rows of every sequence and head, tile edges of the first/last
    query tile, window edges)."""
    rng = np.random.default_rng(seed)
    wl = inp.wl
    H = wl.hq
    rows = set()
    if inp.cu_seqlens is not None:
        T = inp.total_tokens
        total = H * T
        cu = inp.cu_seqlens.tolist()
        for h in {0, H // 2, H - 1}:
            for s in range(len(cu) - 1):
                a, b = cu[s], cu[s + 1]
                for t in {a, a + 1, b - 1, b - 2, a + block_m - 1, a + block_m}:
                    if a <= t < b:
                        rows.add(h * T + t)
    else:
        B, S = inp.q.shape[0], inp.q.shape[2]
        total = B * H * S
        for b in {0, B - 1}:
            for h in {0, H // 2, H - 1}:
                base = (b * H + h) * S
                cand = {0, 1, block_m - 1, block_m, S - block_m, S - 1, S - 2}
                if wl.window_left >= 0:
                    cand |= {wl.window_left - 1, wl.window_left, wl.window_left + 1,
                             S // 2 + wl.window_left}
                # variant edges: prefix / prompt end, test-query start, global
                # positions, segment starts
                for e in (wl.prefix_len, wl.query_start, wl.num_global):
                    if e > 0:
                        cand |= {e - 1, e, e + 1}
                if inp.segment_starts is not None:
                    for st in inp.segment_starts.tolist():
                        cand |= {st - 1, st, st + 1}
                for i in cand:
                    if 0 <= i < S:
                        rows.add(base + i)
    rows |= set(rng.choice(total, size=min(n_random, total), replace=False).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def nan_fill_(t):
    if t.dtype.is_floating_point:
        t.fill_(math.nan)
    return t

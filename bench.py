"""Benchmark of the fused attention forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--also A,B]

A step is one attn_fwd call (the whole fused forward) over one batch of the
seeded synthetic workload, with inputs already resident in HBM. The default
workload is the largest single-GPU configuration: 16 packed causal sequences
of 256..8192 tokens (61,938 in total) with 32 query and 8 key/value heads of
dimension 128. Prints one
JSON line: throughput in TFLOP/s counting only unmasked score entries
(4 * head_dim FLOPs per visible query/key pair per query head), the roofline
of the kernel against the bf16 matrix-core peak, and the CPU oracle timed on a
bounded sample of the same workload on the host cores. Without --workload the
line also carries `other_configs`: the other four headline workloads (fp32
plain, causal, GQA sliding window, ALiBi + soft-cap), each timed after the
reported one with the same warm-up and step counts; `value` stays that of the
default workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2605_05023_amd as attn  # noqa: E402
from paper_2605_05023_amd.workloads import (MASK_CAUSAL, MASK_CAUSAL_BLOCKWISE,  # noqa: E402
                                            MASK_GLOBAL_WINDOW, MASK_NAMES, MASK_PREFIX_LM,
                                            MASK_SHARE_QUESTION, MASK_SLIDING_WINDOW, WORKLOADS,
                                            make_inputs)

METRIC = "attention fwd TFLOP/s (unmasked FLOPs) and % of bf16 MFMA peak, 1 MI355X"
# Dense bf16 matrix-core peak: 256 CUs x 2.4 GHz x 4096 FLOP/clk/CU (the published 2.5 PFLOP/s).
PEAK_BF16_TFLOPS = 2516.6
PEAK_FP32_TFLOPS = 157.3
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2605_05023_amd", "csrc")
# Everything that decides what a launch does: the kernels, the host side that
# chooses the schedule (heads per workgroup, workgroup order, chunking), and
# the ABI header.
KERNEL_SOURCES = sorted(os.path.join("paper_2605_05023_amd", "csrc", f) for f in os.listdir(CSRC)
                        if f.endswith((".hip", ".h", ".cpp"))) + [os.path.join("include", "attn.h")]


def row_counts(inp, S: int) -> np.ndarray:
    """Visible keys of rows 0..S-1 of one sequence of S tokens (Sq == Sk), in
    closed form per mask kind (Appendix A case analyses)."""
    wl = inp.wl
    i = np.arange(S, dtype=np.int64)

    def band(left, right):
        lo = np.zeros(S, np.int64) if left < 0 else np.maximum(0, i - left)
        hi = np.full(S, S - 1, np.int64) if right < 0 else np.minimum(S - 1, i + right)
        return lo, hi

    if wl.mask == MASK_CAUSAL:
        return i + 1
    if wl.mask == MASK_SLIDING_WINDOW:
        lo, hi = band(wl.window_left, wl.window_right)
        return np.maximum(0, hi - lo + 1)
    if wl.mask == MASK_PREFIX_LM:  # keys j < L_p, or j <= i
        return np.maximum(i + 1, min(wl.prefix_len, S))
    if wl.mask == MASK_GLOBAL_WINDOW:  # |i - j| within the window, or i or j in G
        lo, hi = band(wl.window_left, wl.window_right)
        inside = np.maximum(0, hi - lo + 1)
        if wl.global_list:  # listed G: the keys of G outside the row's band
            g = np.asarray([x for x in wl.global_list if x < S], dtype=np.int64)
            in_band = ((g[None, :] >= lo[:, None]) & (g[None, :] <= hi[:, None])).sum(1)
            n = inside + len(g) - in_band
            return np.where(np.isin(i, g), S, n)
        g = min(wl.num_global, S)
        overlap = np.maximum(0, np.minimum(hi, g - 1) - lo + 1)  # globals already in the band
        n = inside + g - overlap
        return np.where(i < g, S, n)
    if wl.mask in (MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE):
        starts = np.asarray(inp.segment_starts.tolist(), dtype=np.int64)
        k = np.searchsorted(starts, i, side="right") - 1  # segment of row i, -1 before s_0
        seg_start = np.where(k >= 0, starts[np.maximum(k, 0)], 0)
        if wl.mask == MASK_SHARE_QUESTION:  # prompt causal; response: prompt + own segment
            prompt = min(int(starts[0]), S)
            return np.where(k < 0, i + 1, prompt + (i - seg_start + 1))
        return np.where(i >= wl.query_start, i + 1, i - seg_start + 1)
    return np.full(S, S, np.int64)


def visible_pairs(inp) -> int:
    """Visible (query, key) pairs summed over query heads and sequences."""
    wl = inp.wl
    lengths = inp.lengths if inp.lengths is not None else [wl.seqlen] * wl.batch
    return int(sum(int(row_counts(inp, S).sum()) for S in lengths if S > 0)) * wl.hq


def algorithmic_bytes(inp) -> int:
    """Bytes the method must move once: Q, K, V in; O and fp32 LSE out."""
    el = inp.q.element_size()
    return (2 * inp.q.numel() + inp.k.numel() + inp.v.numel()) * el + \
        (inp.q.numel() // inp.wl.head_dim) * 4


def kernel_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(workload: str):
    """Bytes per launch from the committed PMC summary (FETCH_SIZE + WRITE_SIZE,
    calibrated against a plain copy), if it was measured on the current library
    sources (else None). The counters count the L2's traffic to the fabric,
    which includes Infinity Cache hits: an upper bound on HBM bytes."""
    path = os.path.join(PROFILES, f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_hash:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"fabric_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_hash():
        return None
    return float(m_bytes.group(1))


def cpu_baseline(inp, flops_per_row_fn, min_seconds: float, max_seconds: float, seed: int):
    """Time the CPU oracle (as it stands) on a seeded random sample of rows."""
    import oracle  # the benchmark's CPU-baseline leg is allowed to run the oracle

    wl = inp.wl
    qn = inp.q.float().numpy()
    kn = inp.k.float().numpy()
    vn = inp.v.float().numpy()
    total_rows = qn.shape[0] * qn.shape[1] if inp.cu_seqlens is not None else \
        qn.shape[0] * qn.shape[1] * qn.shape[2]
    rng = np.random.default_rng(seed)
    order = rng.permutation(total_rows)
    kw = dict(scale=wl.scale, mask=wl.mask, window_left=wl.window_left,
              window_right=wl.window_right, slopes=inp.slopes, softcap=wl.softcap,
              cu_seqlens_q=inp.cu_seqlens, cu_seqlens_k=inp.cu_seqlens,
              **inp.oracle_mask_kwargs())
    oracle.load()
    done, elapsed, flops, batch = 0, 0.0, 0, 256
    while done < total_rows and elapsed < min_seconds:
        rows = order[done:done + batch]
        t0 = time.perf_counter()
        oracle.attention(qn, kn, vn, rows=rows, **kw)
        dt = time.perf_counter() - t0
        elapsed += dt
        flops += flops_per_row_fn(rows)
        done += len(rows)
        if elapsed + 2 * dt > max_seconds:
            break
        batch = min(batch * 2, 16384)
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f
                              if ln.startswith("model name")), None)
    except OSError:
        pass
    return {
        "value": flops / elapsed / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "cpu_model": cpu_model,
        "kind": "oracle",
        "sample": f"{done} of {total_rows} query rows (seeded random), fp64 dense "
                  f"materialised scores, {elapsed:.1f} s; unit counts unmasked FLOPs of the "
                  f"sampled rows",
    }


def row_flops_fn(inp):
    """Unmasked FLOPs of given flat LSE row ids."""
    wl = inp.wl
    D = wl.head_dim
    if inp.cu_seqlens is not None:
        cu = inp.cu_seqlens.numpy().astype(np.int64)
        T = inp.total_tokens
        counts = [row_counts(inp, int(cu[s + 1] - cu[s])) for s in range(len(cu) - 1)]

        def per_row(rows):
            t = rows % T
            s = np.searchsorted(cu, t, side="right") - 1
            return np.array([counts[a][b] for a, b in zip(s, t - cu[s])], dtype=np.int64)
    else:
        counts = row_counts(inp, wl.seqlen)

        def per_row(rows):
            return counts[rows % wl.seqlen]

    def fn(rows):
        return int(4 * D * per_row(np.asarray(rows, dtype=np.int64)).sum())
    return fn


DEFAULT_WORKLOAD = "varlen_gqa_bf16"
# the workloads the metric is quoted on: fp32 plain, causal, GQA window,
# ALiBi + soft-cap, packed variable-length causal GQA
HEADLINE = ("plain_fp32", "causal_bf16", "gqa_swa_bf16", "alibi_softcap_bf16", "varlen_gqa_bf16")


def time_other(name: str, steps: int, warmup: int, dev) -> dict:
    """One further workload, timed like the reported one: `warmup` launches,
    then `steps` launches between HIP events on the launching stream and the
    host clock. Its inputs are freed afterwards."""
    wl = WORKLOADS[name]
    inp = make_inputs(wl)
    q, k, v = inp.q.to(dev), inp.k.to(dev), inp.v.to(dev)
    out = torch.empty_like(q)
    varlen = inp.cu_seqlens is not None
    lse_shape = (wl.hq, inp.total_tokens) if varlen else (wl.batch, wl.hq, wl.seqlen)
    lse = torch.empty(lse_shape, dtype=torch.float32, device=dev) if wl.norm == "softmax" else None
    vkw = inp.variant_kwargs(dev)
    stream = torch.cuda.current_stream(dev)
    desc = attn.make_desc(q, k, v, out, stream=stream.cuda_stream, **vkw)
    lib = attn.load()
    args_c = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
              lse.data_ptr() if lse is not None else None, ctypes.byref(desc))
    for _ in range(warmup):
        attn.check(lib.attn_fwd(*args_c), lib)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        attn.check(lib.attn_fwd(*args_c), lib)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kernel_ms = e0.elapsed_time(e1) / steps
    flops = 4 * wl.head_dim * visible_pairs(inp)
    ms_per_step = wall * 1e3 / steps
    value = flops / (ms_per_step * 1e-3) / 1e12
    achieved = flops / (kernel_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    return {
        "workload": name,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "value": round(value, 2),
        "ms_per_step": round(ms_per_step, 5),
        "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "kernel_avg_ms": round(kernel_ms, 5),
        "achieved": round(achieved, 2),
        "peak": peak,
        "frac": round(achieved / peak, 4),
        "unmasked_flops_per_step": flops,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None, choices=sorted(WORKLOADS),
                    help="workload of the reported value (default varlen_gqa_bf16)")
    ap.add_argument("--also", default=None,
                    help="comma-separated further workloads timed after the reported one, in the "
                         "same way, into other_configs (default: the other headline workloads "
                         "when --workload is not given, none otherwise; 'none' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="minimum oracle time for the CPU baseline sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one 1 GiB device copy (counter calibration under rocprofv3)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the benchmark measures one MI355X "
              f"(the kernel on one GPU's share); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)

    also = args.also
    if args.workload is None:
        args.workload = DEFAULT_WORKLOAD
        if also is None:
            also = ",".join(w for w in HEADLINE if w != DEFAULT_WORKLOAD)
    also = [] if also in (None, "", "none") else also.split(",")
    for w in also:
        if w not in WORKLOADS:
            print(f"bench.py: unknown workload {w} in --also", file=sys.stderr)
            sys.exit(2)

    dev = torch.device("cuda:0")
    wl = WORKLOADS[args.workload]
    inp = make_inputs(wl)
    q, k, v = inp.q.to(dev), inp.k.to(dev), inp.v.to(dev)
    out = torch.empty_like(q)
    varlen = inp.cu_seqlens is not None
    lse_shape = (wl.hq, inp.total_tokens) if varlen else (wl.batch, wl.hq, wl.seqlen)
    lse = torch.empty(lse_shape, dtype=torch.float32, device=dev) if wl.norm == "softmax" else None
    vkw = inp.variant_kwargs(dev)  # keeps the device copies of slopes / segments alive
    stream = torch.cuda.current_stream(dev)
    desc = attn.make_desc(q, k, v, out, stream=stream.cuda_stream, **vkw)
    lib = attn.load()
    args_c = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
              lse.data_ptr() if lse is not None else None, ctypes.byref(desc))

    def step():
        rc = lib.attn_fwd(*args_c)
        if rc != 0:
            attn.check(rc, lib)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kernel_ms = e0.elapsed_time(e1) / args.steps

    # Per-launch durations, outside the timed region, from HIP events queued
    # around each launch on the same stream (no host wait in between): launches
    # with warm caches alternate with launches after a 512 MiB write that
    # evicts the inputs from the L2s and the 256 MB Infinity Cache, so that the
    # drift of the power-limited clock under sustained load affects both alike.
    reps = max(1, min(args.steps, 30))
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
    for w0, w1, c0, c1 in ev:
        w0.record(stream)
        step()
        w1.record(stream)
        flush.fill_(0)
        c0.record(stream)
        step()
        c1.record(stream)
    torch.cuda.synchronize()
    warm = sorted(w0.elapsed_time(w1) for w0, w1, _, _ in ev)
    cold = sorted(c0.elapsed_time(c1) for _, _, c0, c1 in ev)
    del flush

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    flops = 4 * wl.head_dim * visible_pairs(inp)
    ms_per_step = wall * 1e3 / args.steps
    value = flops / (ms_per_step * 1e-3) / 1e12
    achieved = flops / (kernel_ms * 1e-3) / 1e12
    # bf16 runs on the matrix cores; the fp32 kernel computes on the vector ALUs
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    nbytes = algorithmic_bytes(inp)
    traffic = read_traffic(args.workload)

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0, sigma^2) inputs; no dataset)",
        "config": {
            "workload": args.workload,
            "batch": wl.batch,
            "heads_q": wl.hq,
            "heads_kv": wl.hkv,
            "seqlen": wl.seqlen if not varlen else f"varlen, total {inp.total_tokens}",
            "head_dim": wl.head_dim,
            "mask": MASK_NAMES[wl.mask],
            "window": [wl.window_left, wl.window_right]
            if wl.mask in (MASK_SLIDING_WINDOW, MASK_GLOBAL_WINDOW) else None,
            "alibi": wl.alibi,
            "softcap": wl.softcap,
            "relative_position": wl.relpos,
            "norm": wl.norm,
            "prefix_len": wl.prefix_len if wl.mask in (MASK_PREFIX_LM, MASK_SHARE_QUESTION) else None,
            "num_global": wl.num_global if wl.mask == MASK_GLOBAL_WINDOW else None,
            "global_list": list(wl.global_list) if wl.global_list else None,
            "segment_starts": inp.segment_starts.tolist() if inp.segment_starts is not None else None,
            "query_start": wl.query_start if wl.mask == MASK_CAUSAL_BLOCKWISE else None,
            "unmasked_flops_per_step": flops,
        },
        "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": {
            "bound": "mfma" if wl.dtype == "bf16" else "alu",
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": traffic,
            "kernel_avg_ms": round(kernel_ms, 5),
            "kernel_median_ms": round(warm[len(warm) // 2], 5),
            "kernel_min_ms": round(warm[0], 5),
            "kernel_max_ms": round(warm[-1], 5),
            "kernel_cold_median_ms": round(cold[len(cold) // 2], 5),
            "algorithmic_bytes": nbytes,
            "algorithmic_gbps": round(nbytes / (kernel_ms * 1e-3) / 1e9, 1),
        },
    }
    if also:
        del q, k, v, out, lse, vkw, desc
        result["other_configs"] = [time_other(w, args.steps, args.warmup, dev) for w in also]
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(inp, row_flops_fn(inp), args.cpu_seconds,
                                              4 * args.cpu_seconds, seed=wl.seed)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

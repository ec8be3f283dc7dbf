"""bench.py's closed-form count of visible (query, key) pairs -- the FLOP
numerator of every reported TFLOP/s -- against the CPU oracle's mask (with
zero queries P > 0 exactly on visible pairs), for every mask kind."""
import dataclasses
import os
import sys

import numpy as np
import pytest
import torch

import oracle

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402
from paper_2605_05023_amd.workloads import WORKLOADS, make_inputs  # noqa: E402

NAMES = ["causal_bf16", "gqa_swa_bf16", "alibi_softcap_bf16", "prefixlm_bf16",
         "global_window_bf16", "global_window_listed_bf16", "share_question_bf16",
         "causal_blockwise_bf16", "relu_bf16"]


@pytest.mark.parametrize("name", NAMES)
def test_row_counts_match_oracle_mask(name):
    wl = WORKLOADS[name]
    for S in (1, 37, 300):
        small = dataclasses.replace(
            wl, seqlen=S, batch=1, hq=1, hkv=1, prefix_len=min(wl.prefix_len, S // 3),
            query_start=min(wl.query_start, 2 * S // 3), num_global=min(wl.num_global, 5),
            window_left=min(wl.window_left, 20) if wl.window_left >= 0 else -1,
            window_right=min(wl.window_right, 20) if wl.window_right >= 0 else -1)
        inp = make_inputs(small)
        kw = inp.oracle_mask_kwargs()
        kw["norm"] = oracle.NORM_SOFTMAX
        q = torch.zeros((1, 1, S, 4))
        kv = torch.ones((1, 1, S, 4))
        _, _, p = oracle.attention(q, kv, kv, scale=1.0, mask=small.mask,
                                   window_left=small.window_left,
                                   window_right=small.window_right, want_probs=True, **kw)
        assert np.array_equal((p[0, 0] > 0).sum(1), bench.row_counts(inp, S)), (name, S)


def test_headline_pair_counts():
    # causal S(S+1)/2 x 64 heads; window: sum_i min(i+1, 1024) x 64 heads
    assert bench.visible_pairs(make_inputs(WORKLOADS["causal_bf16"])) == 2048 * 2049 // 2 * 64
    assert bench.visible_pairs(make_inputs(WORKLOADS["gqa_swa_bf16"])) == \
        sum(min(i + 1, 1024) for i in range(8192)) * 64


TRAFFIC = sorted(f[len("traffic_"):-3] for f in os.listdir(bench.PROFILES)
                 if f.startswith("traffic_") and f.endswith(".md"))


def _field(text, key):
    import re
    m = re.search(rf"{key}:\s*([0-9a-fA-F.eE+]+)", text)
    assert m, key
    return m.group(1)


@pytest.mark.parametrize("name", TRAFFIC)
def test_traffic_summary(name):
    """Each committed memory-traffic summary names a workload, states no fewer
    bytes than the method must move, and is used by bench.py only while its
    library-source hash is the current one."""
    assert name in WORKLOADS
    text = open(os.path.join(bench.PROFILES, f"traffic_{name}.md")).read()
    hbm = float(_field(text, "fabric_bytes_per_launch"))
    alg = int(_field(text, "algorithmic_bytes_per_launch"))
    assert hbm >= 0.9 * alg
    if name == "causal_bf16":
        assert alg == bench.algorithmic_bytes(make_inputs(WORKLOADS[name]))
    stored = _field(text, "kernel_hash")
    current = bench.kernel_hash()
    assert bench.read_traffic(name) == (hbm if stored == current else None)


def test_grid_pair_counts():
    """The paper-grid workloads (16k tokens, 128 query heads): causal rows see
    i + 1 keys, window rows min(i + 1, 1024)."""
    import types
    from paper_2605_05023_amd.workloads import GRID_ORDER, MASK_SLIDING_WINDOW
    for name in GRID_ORDER:
        wl = WORKLOADS[name]
        S = wl.seqlen
        per_seq = sum(min(i + 1, 1024) for i in range(S)) if wl.mask == MASK_SLIDING_WINDOW \
            else S * (S + 1) // 2
        inp = types.SimpleNamespace(wl=wl, lengths=None, segment_starts=None)
        assert wl.batch * S == 16384 and (wl.hq, wl.hkv, wl.head_dim) == (128, 8, 128)
        assert bench.visible_pairs(inp) == per_seq * wl.batch * 128, name

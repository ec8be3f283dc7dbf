"""GPU parity for the further variants of Appendix A: PrefixLM, the relative
position term, ReLU and Sigmoid normalisation (and the PrefixLM + soft-cap +
Sigmoid combination), the global sliding window, the share question mask and
the causal blockwise mask, through the C ABI against the CPU oracle.

Small cases compare every output element, span several query and key tiles
with ragged tails, and cover both kernel paths (closed-form band masks and
the general per-row path), both head dims, grouped-query heads, varlen and
fp32. The full-size workloads compare seeded samples of rows plus the
variant's edges (4096 seeded rows of the 524,288: the oracle takes a minute
per workload for all of them). Bars: softmax O max-abs 2e-2 (bf16) / 1e-4 (fp32) and LSE
1e-3; ReLU / Sigmoid O within that fraction of max|O_ref| (no LSE).
"""
import numpy as np
import pytest

from gpu_util import assert_parity, gpu_available, log, run_gpu, sample_rows
from paper_2605_05023_amd.workloads import (MASK_CAUSAL, MASK_CAUSAL_BLOCKWISE, MASK_GLOBAL_WINDOW,
                                            MASK_NONE, MASK_PREFIX_LM, MASK_SHARE_QUESTION,
                                            MASK_SLIDING_WINDOW, NEXT_ORDER, WORKLOADS, Workload,
                                            make_inputs)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def W(name, dtype, B, hq, hkv, S, D, mask=MASK_NONE, seed=21, **kw):
    return Workload(name, dtype, B, hq, hkv, S, D, mask=mask, seed=seed, **kw)


SMALL = [
    # PrefixLM (closed-form band path)
    W("prefix_d128", "bf16", 2, 2, 2, 300, 128, MASK_PREFIX_LM, prefix_len=100),
    W("prefix_d128_lp0", "bf16", 1, 2, 2, 200, 128, MASK_PREFIX_LM, prefix_len=0),
    W("prefix_d128_lp1", "bf16", 1, 2, 2, 200, 128, MASK_PREFIX_LM, prefix_len=1),
    W("prefix_d128_all", "bf16", 1, 2, 2, 150, 128, MASK_PREFIX_LM, prefix_len=150),
    W("prefix_d64_gqa", "bf16", 2, 4, 2, 333, 64, MASK_PREFIX_LM, prefix_len=77),
    W("prefix_d128_tile_edge", "bf16", 1, 2, 2, 256, 128, MASK_PREFIX_LM, prefix_len=128),
    # relative position (closed-form path; general path when combined with ALiBi)
    W("relpos_causal_d128", "bf16", 2, 2, 2, 300, 128, MASK_CAUSAL, relpos=True),
    W("relpos_none_d64", "bf16", 1, 3, 3, 200, 64, relpos=True),
    W("relpos_window_d128", "bf16", 1, 2, 2, 300, 128, MASK_SLIDING_WINDOW, window_left=40,
      window_right=0, relpos=True),
    W("relpos_softcap_d64", "bf16", 1, 2, 2, 260, 64, MASK_CAUSAL, relpos=True, softcap=20.0),
    W("relpos_alibi_d128", "bf16", 1, 4, 4, 200, 128, MASK_CAUSAL, relpos=True, alibi=True),
    W("relpos_prefix_d128", "bf16", 1, 2, 2, 220, 128, MASK_PREFIX_LM, prefix_len=60,
      relpos=True),
    # ReLU / Sigmoid normalisation and the combination
    W("relu_causal_d128", "bf16", 2, 2, 2, 300, 128, MASK_CAUSAL, norm="relu"),
    W("relu_none_d64", "bf16", 1, 3, 3, 257, 64, norm="relu"),
    W("relu_alibi_softcap_d128", "bf16", 1, 4, 2, 200, 128, MASK_CAUSAL, norm="relu",
      alibi=True, softcap=30.0),
    W("relu_relpos_d64", "bf16", 1, 2, 2, 150, 64, MASK_CAUSAL, norm="relu", relpos=True),
    W("sigmoid_causal_d128", "bf16", 2, 2, 2, 300, 128, MASK_CAUSAL, norm="sigmoid"),
    W("sigmoid_window_d64", "bf16", 1, 2, 2, 280, 64, MASK_SLIDING_WINDOW, norm="sigmoid",
      window_left=50, window_right=10),
    W("combo_d128", "bf16", 2, 2, 2, 300, 128, MASK_PREFIX_LM, prefix_len=90, softcap=50.0,
      norm="sigmoid", sigma=1.5),
    W("combo_d64_gqa", "bf16", 1, 4, 1, 260, 64, MASK_PREFIX_LM, prefix_len=130, softcap=20.0,
      norm="sigmoid"),
    # global sliding window (general path)
    W("global_d128", "bf16", 2, 2, 2, 300, 128, MASK_GLOBAL_WINDOW, window_left=20,
      window_right=20, num_global=5),
    W("global_d128_w0_g1", "bf16", 1, 2, 2, 200, 128, MASK_GLOBAL_WINDOW, window_left=0,
      window_right=0, num_global=1),
    W("global_d64_g0", "bf16", 1, 2, 2, 260, 64, MASK_GLOBAL_WINDOW, window_left=30,
      window_right=30, num_global=0),
    W("global_d128_wide_g", "bf16", 1, 2, 2, 333, 128, MASK_GLOBAL_WINDOW, window_left=8,
      window_right=64, num_global=140),
    # global sliding window with a listed global set (gathered tiles): scattered
    # positions, positions inside and outside the band, a tile-sized run, the
    # last key, positions past the end, a single entry
    W("glist_d128", "bf16", 2, 2, 2, 300, 128, MASK_GLOBAL_WINDOW, window_left=20,
      window_right=20, global_list=(0, 5, 150, 299)),
    W("glist_d64_gqa_one_sided", "bf16", 2, 8, 2, 333, 64, MASK_GLOBAL_WINDOW, window_left=40,
      window_right=0, global_list=(3, 64, 65, 200, 330, 500)),
    W("glist_d128_run_of_70", "bf16", 1, 4, 4, 400, 128, MASK_GLOBAL_WINDOW, window_left=8,
      window_right=8, global_list=tuple(range(100, 170)) + (399,)),
    # grouped heads (32 rows per workgroup): 70 global rows take three chunks of
    # the list, the last one partial, and a position past the end is ignored
    W("glist_d128_gqa4_three_chunks", "bf16", 2, 8, 2, 300, 128, MASK_GLOBAL_WINDOW,
      window_left=12, window_right=3, global_list=tuple(range(5, 285, 4)) + (299, 400)),
    W("glist_d128_single_w0", "bf16", 1, 2, 2, 200, 128, MASK_GLOBAL_WINDOW, window_left=0,
      window_right=0, global_list=(77,)),
    W("glist_d64_alibi_relpos_softcap", "bf16", 1, 4, 4, 260, 64, MASK_GLOBAL_WINDOW,
      window_left=16, window_right=16, global_list=(1, 128, 250), alibi=True, relpos=True,
      softcap=30.0, sigma=1.5),
    W("glist_d128_relpos", "bf16", 1, 2, 2, 300, 128, MASK_GLOBAL_WINDOW, window_left=10,
      window_right=5, global_list=(2, 100, 290), relpos=True),
    W("glist_d128_sigmoid", "bf16", 1, 2, 2, 300, 128, MASK_GLOBAL_WINDOW, window_left=30,
      window_right=30, global_list=(0, 64, 200), norm="sigmoid"),
    W("glist_d64_relu_softcap", "bf16", 1, 3, 3, 220, 64, MASK_GLOBAL_WINDOW, window_left=12,
      window_right=12, global_list=(10, 11, 190), norm="relu", softcap=20.0),
    W("fp32_glist", "fp32", 1, 2, 2, 150, 64, MASK_GLOBAL_WINDOW, window_left=10,
      window_right=10, global_list=(4, 70, 149)),
    W("fp32_glist_d128_relpos", "fp32", 1, 2, 2, 130, 128, MASK_GLOBAL_WINDOW, window_left=5,
      window_right=5, global_list=(0, 40, 41, 100), relpos=True),
    # share question (general path)
    W("share_d128", "bf16", 2, 2, 2, 300, 128, MASK_SHARE_QUESTION, prefix_len=64,
      num_segments=3),
    W("share_d128_no_prompt", "bf16", 1, 2, 2, 260, 128, MASK_SHARE_QUESTION, prefix_len=0,
      num_segments=4),
    W("share_d64_gqa", "bf16", 1, 4, 2, 400, 64, MASK_SHARE_QUESTION, prefix_len=150,
      num_segments=5),
    W("share_d128_relpos_softcap", "bf16", 1, 2, 2, 300, 128, MASK_SHARE_QUESTION,
      prefix_len=100, num_segments=2, relpos=True, softcap=30.0),
    # causal blockwise (general path)
    W("blockwise_d128", "bf16", 2, 2, 2, 300, 128, MASK_CAUSAL_BLOCKWISE, num_segments=4,
      query_start=200),
    W("blockwise_d128_lq0", "bf16", 1, 2, 2, 200, 128, MASK_CAUSAL_BLOCKWISE, num_segments=3,
      query_start=0),
    W("blockwise_d64_no_query", "bf16", 1, 3, 3, 300, 64, MASK_CAUSAL_BLOCKWISE,
      num_segments=6, query_start=300),
    W("blockwise_d128_sigmoid", "bf16", 1, 2, 2, 260, 128, MASK_CAUSAL_BLOCKWISE,
      num_segments=4, query_start=180, norm="sigmoid"),
    # fp32 kernel
    W("fp32_prefix", "fp32", 1, 2, 2, 150, 64, MASK_PREFIX_LM, prefix_len=40),
    W("fp32_relpos_causal", "fp32", 1, 2, 2, 130, 128, MASK_CAUSAL, relpos=True),
    W("fp32_relu", "fp32", 1, 2, 2, 120, 64, MASK_CAUSAL, norm="relu"),
    W("fp32_combo", "fp32", 1, 2, 2, 140, 64, MASK_PREFIX_LM, prefix_len=33, softcap=50.0,
      norm="sigmoid"),
    W("fp32_global", "fp32", 1, 2, 2, 150, 64, MASK_GLOBAL_WINDOW, window_left=10,
      window_right=10, num_global=3),
    W("fp32_share", "fp32", 1, 2, 2, 160, 128, MASK_SHARE_QUESTION, prefix_len=40,
      num_segments=3),
    W("fp32_blockwise", "fp32", 1, 2, 2, 170, 64, MASK_CAUSAL_BLOCKWISE, num_segments=4,
      query_start=120),
]


@pytest.mark.parametrize("wl", SMALL, ids=[w.name for w in SMALL])
def test_small_next(wl):
    inp = make_inputs(wl)
    log(f"[next small] {wl.name}: B={wl.batch} Hq={wl.hq} Hkv={wl.hkv} S={wl.seqlen} "
        f"D={wl.head_dim} mask={wl.mask} norm={wl.norm} seg={None if inp.segment_starts is None else inp.segment_starts.tolist()}")
    o, lse = run_gpu(inp)
    assert_parity(inp, o, lse, label=wl.name)


VARLEN = [
    W("varlen_prefix", "bf16", 4, 4, 2, 0, 128, MASK_PREFIX_LM, prefix_len=50),
    # listed global positions are per sequence; those past a sequence's end are ignored
    W("varlen_glist", "bf16", 4, 4, 2, 0, 128, MASK_GLOBAL_WINDOW, window_left=16,
      window_right=16, global_list=(0, 6, 129, 250)),
    W("varlen_glist_fp32", "fp32", 4, 2, 2, 0, 64, MASK_GLOBAL_WINDOW, window_left=8,
      window_right=8, global_list=(3, 100, 200)),
    W("varlen_share", "bf16", 3, 2, 2, 0, 128, MASK_SHARE_QUESTION, prefix_len=40,
      num_segments=3),
    W("varlen_relu_relpos", "bf16", 3, 4, 4, 0, 64, MASK_CAUSAL, norm="relu", relpos=True),
]


@pytest.mark.parametrize("wl", VARLEN, ids=[w.name for w in VARLEN])
def test_varlen_next(wl):
    import dataclasses
    wl = dataclasses.replace(wl, varlen=True)
    inp = make_inputs(wl, lengths=[130, 0, 300, 7][:wl.batch])
    log(f"[next varlen] {wl.name}: lengths={inp.lengths}")
    o, lse = run_gpu(inp)
    assert_parity(inp, o, lse, label=wl.name)


@pytest.mark.parametrize("name", NEXT_ORDER)
def test_full_next(name):
    inp = make_inputs(WORKLOADS[name])
    rows = sample_rows(inp, 4096, seed=3)
    wl = inp.wl
    if wl.global_list:  # every row of the listed global set, in every head
        S = wl.seqlen
        g = [x for x in wl.global_list if x < S]
        extra = [(b * wl.hq + h) * S + x for b in range(wl.batch) for h in range(wl.hq) for x in g]
        rows = np.unique(np.concatenate([np.asarray(rows, dtype=np.int64), extra]))
    log(f"[next full] {name}: {len(rows)} sampled rows")
    o, lse = run_gpu(inp)
    assert_parity(inp, o, lse, rows=rows, label=name)

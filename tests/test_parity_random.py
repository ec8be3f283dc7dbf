"""GPU parity on seeded random variant combinations.

Three batches of 48 configurations, each drawn once from a fixed seed:
dtype, head dim, batch, group size and kv heads, length (fixed or packed
varlen), every mask kind with random bounds, ALiBi, the relative position
term, soft-cap values on both sides of the short form's limit, and the three
normalisations. Each compares every output element with the CPU oracle at
the bars of the other parity tests. They exercise combinations no
hand-written case lists (head-set packing with window and prefix masks,
varlen with the index masks, soft-cap with ReLU, ...).
"""
import numpy as np
import pytest

from gpu_util import assert_parity, gpu_available, log, run_gpu
from paper_2605_05023_amd.workloads import (MASK_CAUSAL, MASK_CAUSAL_BLOCKWISE, MASK_GLOBAL_WINDOW,
                                            MASK_NAMES, MASK_NONE, MASK_PREFIX_LM,
                                            MASK_SHARE_QUESTION, MASK_SLIDING_WINDOW, Workload,
                                            make_inputs)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

MASKS = [MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW, MASK_PREFIX_LM, MASK_GLOBAL_WINDOW,
         MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE]


def _draw_cases(n=48, seed=2605):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        dtype = "fp32" if rng.random() < 0.15 else "bf16"
        D = int(rng.choice([64, 128]))
        group = int(rng.choice([1, 2, 3, 4, 8]))
        hkv = int(rng.integers(1, 3))
        hq = group * hkv
        B = int(rng.integers(1, 4))
        varlen = rng.random() < 0.3
        S = int(rng.integers(1, 321))
        mask = MASKS[int(rng.integers(0, len(MASKS)))]
        kw = {}
        if mask in (MASK_SLIDING_WINDOW, MASK_GLOBAL_WINDOW):
            kw["window_left"] = int(rng.choice([-1, int(rng.integers(0, 200))]))
            kw["window_right"] = int(rng.choice([-1, 0, int(rng.integers(0, 60))]))
            if mask == MASK_GLOBAL_WINDOW:
                kw["num_global"] = int(rng.integers(1, 20))
        if mask == MASK_PREFIX_LM:
            kw["prefix_len"] = int(rng.integers(0, S + 1))
        if mask == MASK_SHARE_QUESTION:
            kw["prefix_len"] = int(rng.integers(1, max(2, S // 2)))
            kw["num_segments"] = int(rng.integers(1, 5))
        if mask == MASK_CAUSAL_BLOCKWISE:
            kw["query_start"] = int(rng.integers(1, S + 1))
            kw["num_segments"] = int(rng.integers(1, 6))
        norm = str(rng.choice(["softmax"] * 8 + ["relu", "sigmoid"]))
        alibi = rng.random() < 0.25
        relpos = rng.random() < 0.15
        softcap = float(rng.choice([0.0] * 6 + [5.0, 30.0, 50.0, 300.0, 1e4]))
        sigma = 1.5 if (alibi or softcap) else 1.0
        name = (f"s{seed}_r{i:02d}_{dtype}_d{D}_g{group}x{hkv}_b{B}_{'varlen' if varlen else f's{S}'}"
                f"_{MASK_NAMES[mask]}{'_alibi' if alibi else ''}{'_relpos' if relpos else ''}"
                f"{f'_cap{softcap:g}' if softcap else ''}{'' if norm == 'softmax' else '_' + norm}")
        wseed = int(rng.integers(0, 1 << 30))
        if mask == MASK_GLOBAL_WINDOW:
            # half of them list G instead (sorted positions, some past the end),
            # drawn from the case's own generator so the other cases stay put
            g = np.random.default_rng(wseed + 1)
            if g.random() < 0.5:
                n = int(g.integers(1, 12))
                kw["global_list"] = tuple(sorted(g.choice(S + 20, size=min(n, S + 20),
                                                          replace=False).tolist()))
                name += "_listed"
        wl = Workload(name, dtype, B, hq, hkv, 0 if varlen else S, D, mask=mask, alibi=alibi,
                      relpos=relpos, softcap=softcap, norm=norm, sigma=sigma,
                      seed=wseed, varlen=varlen, len_lo=0, len_hi=S, **kw)
        cases.append(wl)
    return cases


CASES = _draw_cases(48, 2605) + _draw_cases(48, 7) + _draw_cases(48, 11)


@pytest.mark.parametrize("wl", CASES, ids=[w.name for w in CASES])
def test_random_case(wl):
    inp = make_inputs(wl)
    log(f"[parity random] {wl.name} lengths={inp.lengths}")
    o, lse = run_gpu(inp)
    assert_parity(inp, o, lse, label=wl.name)

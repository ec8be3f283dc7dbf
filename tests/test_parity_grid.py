"""GPU parity on the shape grid of the paper's comparison with a hand-written
library (Section 4.1, Appendix C): the Llama3.1-405B attention tuple
128/8/128 (16 query heads per kv head) at S = 1k, 2k, 4k and 8k with 16k
tokens per batch, for the causal, sliding-window (1023, 0), causal soft-cap
(C = 50) and causal ALiBi variants, through the C ABI against the CPU oracle.

Each workload compares 1024 seeded random rows plus the structural ones
(first and last rows of sampled heads, tile and window edges): the oracle on
all 2M rows of a workload would take minutes. Bars: O max-abs 2e-2, LSE 1e-3.
"""
import pytest

from gpu_util import assert_parity, gpu_available, log, run_gpu, sample_rows
from paper_2605_05023_amd.workloads import GRID_ORDER, WORKLOADS, make_inputs

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


@pytest.mark.parametrize("name", GRID_ORDER)
def test_grid_sampled(name):
    inp = make_inputs(WORKLOADS[name])
    rows = sample_rows(inp, 1024, seed=5)
    wl = inp.wl
    log(f"[grid] {name}: B={wl.batch} Hq={wl.hq} Hkv={wl.hkv} S={wl.seqlen}, {len(rows)} rows")
    o, lse = run_gpu(inp)
    assert_parity(inp, o, lse, rows=rows, label=name)

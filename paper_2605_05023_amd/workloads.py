"""Seeded synthetic workloads for the attention forward pass.

This module only describes shapes and draws random inputs. It holds none of
the attention arithmetic, so both the HIP path and the CPU oracle can take
their inputs from here without sharing any of the method.

The paper measures on model-shaped random tensors (Section 4.1, "Benchmark
Configurations": head tuples query/kv/head-dim such as 32/32/128, 64/8/128,
128/8/128, sequence lengths 1k-8k at 16k tokens per batch) and fixes no value
distribution. The five workloads below keep that shape family and add the
variants of Appendix A that this library implements.

Input recipe (identical on every machine because it uses the CPU generator):
    g = torch.Generator().manual_seed(seed)
    varlen only: lengths = torch.randint(lo, hi + 1, (nseq,), generator=g)
    q, k, v = torch.randn(shape, generator=g) * sigma, drawn in that order
    bf16 workloads round the fp32 draw to bfloat16 (round-to-nearest-even).
ALiBi slopes are inputs too: slope_h = 2 ** (-8 h / H) for h = 1..H.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

MASK_NONE = 0
MASK_CAUSAL = 1
MASK_SLIDING_WINDOW = 2


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                 # "bf16" or "fp32"
    batch: int                 # B, or number of sequences when varlen
    hq: int
    hkv: int
    seqlen: int                # S for fixed-length workloads (Sq == Sk)
    head_dim: int
    mask: int = MASK_NONE
    window_left: int = -1
    window_right: int = -1
    alibi: bool = False
    softcap: float = 0.0
    sigma: float = 1.0
    seed: int = 0
    varlen: bool = False
    len_lo: int = 0            # varlen: lengths uniform in [len_lo, len_hi]
    len_hi: int = 0

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


WORKLOADS = {
    # plain softmax attention, fp32, B=1 H=2 S=128 D=64
    "plain_fp32": Workload("plain_fp32", "fp32", 1, 2, 2, 128, 64, seed=0),
    # causal, bf16, B=4 H=16 S=2048 D=128
    "causal_bf16": Workload("causal_bf16", "bf16", 4, 16, 16, 2048, 128,
                            mask=MASK_CAUSAL, seed=1),
    # grouped-query causal sliding window (keys i-1023..i), B=2 Hq=32 Hkv=8 S=8192 D=128
    "gqa_swa_bf16": Workload("gqa_swa_bf16", "bf16", 2, 32, 8, 8192, 128,
                             mask=MASK_SLIDING_WINDOW, window_left=1023,
                             window_right=0, seed=2),
    # non-causal, ALiBi + tanh soft-cap 50, B=8 H=16 S=4096 D=64, sigma 1.5
    "alibi_softcap_bf16": Workload("alibi_softcap_bf16", "bf16", 8, 16, 16, 4096, 64,
                                   alibi=True, softcap=50.0, sigma=1.5, seed=3),
    # variable-length packed causal GQA, 16 sequences of 256..8192 tokens
    "varlen_gqa_bf16": Workload("varlen_gqa_bf16", "bf16", 16, 32, 8, 0, 128,
                                mask=MASK_CAUSAL, seed=4, varlen=True,
                                len_lo=256, len_hi=8192),
}

# Order used when a list of all five is wanted.
WORKLOAD_ORDER = ["plain_fp32", "causal_bf16", "gqa_swa_bf16",
                  "alibi_softcap_bf16", "varlen_gqa_bf16"]


@dataclasses.dataclass
class Inputs:
    """Host tensors for one workload. Layouts: fixed length q/o [B,Hq,S,D],
    k/v [B,Hkv,S,D]; varlen q/o [T,Hq,D], k/v [T,Hkv,D] with cu_seqlens."""
    wl: Workload
    q: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    slopes: Optional[torch.Tensor]       # fp32 [Hq] or None
    cu_seqlens: Optional[torch.Tensor]   # int32 [B+1] or None
    lengths: Optional[list]

    @property
    def max_seqlen(self) -> int:
        if self.lengths is None:
            return self.wl.seqlen
        return max(self.lengths) if self.lengths else 0

    @property
    def total_tokens(self) -> int:
        if self.lengths is None:
            return self.wl.batch * self.wl.seqlen
        return sum(self.lengths)


def alibi_slopes(nheads: int) -> torch.Tensor:
    """slope_h = 2^(-8h/H), h = 1..H, as fp32 (an input of the ALiBi variant)."""
    return torch.tensor([2.0 ** (-8.0 * h / nheads) for h in range(1, nheads + 1)],
                        dtype=torch.float32)


def cu_from_lengths(lengths) -> torch.Tensor:
    cu = [0]
    for n in lengths:
        cu.append(cu[-1] + int(n))
    return torch.tensor(cu, dtype=torch.int32)


def _draw(shape, g, sigma, dtype):
    x = torch.randn(shape, dtype=torch.float32, generator=g) * sigma
    if dtype == "bf16":
        x = x.to(torch.bfloat16)
    return x


def make_inputs(wl: Workload, *, lengths=None, seqlen=None, batch=None,
                seed=None) -> Inputs:
    """Draw the seeded inputs of `wl`. `lengths`, `seqlen`, `batch` and `seed`
    override the workload's own values (used for small parity cases)."""
    g = torch.Generator().manual_seed(wl.seed if seed is None else seed)
    B = wl.batch if batch is None else batch
    if wl.varlen:
        if lengths is None:
            lengths = torch.randint(wl.len_lo, wl.len_hi + 1, (B,), generator=g).tolist()
        lengths = [int(x) for x in lengths]
        T = sum(lengths)
        qs, ks = (T, wl.hq, wl.head_dim), (T, wl.hkv, wl.head_dim)
        cu = cu_from_lengths(lengths)
    else:
        S = wl.seqlen if seqlen is None else seqlen
        qs, ks = (B, wl.hq, S, wl.head_dim), (B, wl.hkv, S, wl.head_dim)
        cu = None
        lengths = None
    q = _draw(qs, g, wl.sigma, wl.dtype)
    k = _draw(ks, g, wl.sigma, wl.dtype)
    v = _draw(ks, g, wl.sigma, wl.dtype)
    if wl.varlen or seqlen is not None or batch is not None:
        wl = dataclasses.replace(wl, batch=len(lengths) if wl.varlen else B,
                                 seqlen=0 if wl.varlen else (wl.seqlen if seqlen is None else seqlen))
    slopes = alibi_slopes(wl.hq) if wl.alibi else None
    return Inputs(wl, q, k, v, slopes, cu, lengths)

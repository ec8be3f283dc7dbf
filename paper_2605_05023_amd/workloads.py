"""Seeded synthetic workloads for the attention forward pass.

This module only describes shapes and draws random inputs. It holds none of
the attention arithmetic, so both the HIP path and the CPU oracle can take
their inputs from here without sharing any of the method.

The paper measures on model-shaped random tensors (Section 4.1, "Benchmark
Configurations": head tuples query/kv/head-dim such as 32/32/128, 64/8/128,
128/8/128, sequence lengths 1k-8k at 16k tokens per batch) and fixes no value
distribution. The five headline workloads keep that shape family and add the
variants of Appendix A built in first; the further variants (PrefixLM,
relative position, ReLU / Sigmoid normalisation, their combination, global
sliding window, share question, causal blockwise) each get one workload at
the Llama2-7B tuple 32/32/128 with S = 8k and B = 2 (16k tokens). The
`grid405b_*` workloads repeat the paper's comparison grid: the 128/8/128
tuple at S = 1k..8k, 16k tokens per batch, four variants.

Input recipe (identical on every machine because it uses the CPU generator):
    g = torch.Generator().manual_seed(seed)
    varlen only: lengths = torch.randint(lo, hi + 1, (nseq,), generator=g)
    q, k, v = torch.randn(shape, generator=g) * sigma, drawn in that order
    bf16 workloads round the fp32 draw to bfloat16 (round-to-nearest-even).
ALiBi slopes are inputs too: slope_h = 2 ** (-8 h / H) for h = 1..H.
Segment starts (share question, causal blockwise) are drawn after v from the
same generator: num_segments - 1 distinct cut points, sorted, inside the
response region (prompt_len, S) or the document region (0, query_start).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

MASK_NONE = 0
MASK_CAUSAL = 1
MASK_SLIDING_WINDOW = 2
MASK_PREFIX_LM = 3
MASK_GLOBAL_WINDOW = 4
MASK_SHARE_QUESTION = 5
MASK_CAUSAL_BLOCKWISE = 6
MASK_NAMES = {MASK_NONE: "none", MASK_CAUSAL: "causal", MASK_SLIDING_WINDOW: "sliding_window",
              MASK_PREFIX_LM: "prefix_lm", MASK_GLOBAL_WINDOW: "global_sliding_window",
              MASK_SHARE_QUESTION: "share_question", MASK_CAUSAL_BLOCKWISE: "causal_blockwise"}
NORM_CODES = {"softmax": 0, "relu": 1, "sigmoid": 2}


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
    prefix_len: int = 0        # PrefixLM L_p; share question: prompt length
    num_global: int = 0        # global sliding window: positions 0..num_global-1
    global_list: tuple = ()    # global sliding window: G as listed positions (overrides num_global)
    num_segments: int = 0      # share question responses / blockwise documents
    query_start: int = 0       # causal blockwise L_q
    relpos: bool = False       # relative position term (i - j)
    norm: str = "softmax"      # "softmax", "relu" or "sigmoid"

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

def _llama7b(name, seed, **kw):
    return Workload(name, "bf16", 2, 32, 32, 8192, 128, seed=seed, **kw)


# Further variants of Appendix A, one workload each (Llama2-7B tuple, 16k tokens).
NEXT_WORKLOADS = {
    "prefixlm_bf16": _llama7b("prefixlm_bf16", 5, mask=MASK_PREFIX_LM, prefix_len=2048),
    "relpos_bf16": _llama7b("relpos_bf16", 6, mask=MASK_CAUSAL, relpos=True),
    "relu_bf16": _llama7b("relu_bf16", 7, mask=MASK_CAUSAL, norm="relu"),
    "sigmoid_bf16": _llama7b("sigmoid_bf16", 8, mask=MASK_CAUSAL, norm="sigmoid"),
    "combo_bf16": _llama7b("combo_bf16", 9, mask=MASK_PREFIX_LM, prefix_len=2048,
                           softcap=50.0, norm="sigmoid"),
    "global_window_bf16": _llama7b("global_window_bf16", 10, mask=MASK_GLOBAL_WINDOW,
                                   window_left=512, window_right=512, num_global=16),
    # the same window with a scattered global set: a leading token, a few in
    # the middle, the last one
    "global_window_listed_bf16": _llama7b("global_window_listed_bf16", 13,
                                          mask=MASK_GLOBAL_WINDOW, window_left=512,
                                          window_right=512,
                                          global_list=(0, 5, 300, 2049, 4096, 6000, 8191)),
    "share_question_bf16": _llama7b("share_question_bf16", 11, mask=MASK_SHARE_QUESTION,
                                    prefix_len=2048, num_segments=4),
    "causal_blockwise_bf16": _llama7b("causal_blockwise_bf16", 12, mask=MASK_CAUSAL_BLOCKWISE,
                                      num_segments=8, query_start=6144),
}
WORKLOADS.update(NEXT_WORKLOADS)


def _grid405b(variant, seqlen, seed):
    kw = {"causal": dict(mask=MASK_CAUSAL),
          "window": dict(mask=MASK_SLIDING_WINDOW, window_left=1023, window_right=0),
          "softcap": dict(mask=MASK_CAUSAL, softcap=50.0),
          "alibi": dict(mask=MASK_CAUSAL, alibi=True)}[variant]
    name = f"grid405b_{variant}_s{seqlen // 1024}k"
    return name, Workload(name, "bf16", 16384 // seqlen, 128, 8, seqlen, 128, seed=seed, **kw)


# The shape grid of the paper's comparison with a hand-written library
# (Section 4.1 and Appendix C: the Llama3.1-405B attention tuple 128/8/128,
# S = 1k..8k at 16k tokens per batch) for its four variants there. The paper
# states neither the window nor the cap nor a mask for the soft-cap and ALiBi
# rows: window (1023, 0), C = 50 and a causal mask are this module's choices.
GRID_WORKLOADS = dict(_grid405b(v, s, 20 + 4 * i + j)
                      for i, v in enumerate(("causal", "window", "softcap", "alibi"))
                      for j, s in enumerate((1024, 2048, 4096, 8192)))
WORKLOADS.update(GRID_WORKLOADS)

# Order used when a list of the five headline workloads is wanted.
WORKLOAD_ORDER = ["plain_fp32", "causal_bf16", "gqa_swa_bf16",
                  "alibi_softcap_bf16", "varlen_gqa_bf16"]
NEXT_ORDER = list(NEXT_WORKLOADS)
GRID_ORDER = list(GRID_WORKLOADS)


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
    segment_starts: Optional[torch.Tensor] = None  # int32 [num_segments] or None

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

    def variant_kwargs(self, device=None) -> dict:
        """Keyword arguments of paper_2605_05023_amd.fwd / make_desc for this
        workload's variant (tensors moved to `device`)."""
        wl = self.wl
        kw = dict(mask=MASK_NAMES[wl.mask], softcap=wl.softcap, scale=wl.scale,
                  prefix_len=wl.prefix_len, num_global=wl.num_global,
                  query_start=wl.query_start, relative_position=wl.relpos, norm=wl.norm)
        if wl.mask in (MASK_SLIDING_WINDOW, MASK_GLOBAL_WINDOW):
            kw["window"] = (wl.window_left, wl.window_right)
        if self.slopes is not None:
            kw["alibi_slopes"] = self.slopes.to(device) if device is not None else self.slopes
        if self.segment_starts is not None:
            seg = self.segment_starts
            kw["segment_starts"] = seg.to(device) if device is not None else seg
        if wl.global_list:
            g = torch.tensor(wl.global_list, dtype=torch.int32)
            kw["global_tokens"] = g.to(device) if device is not None else g
            kw["num_global"] = 0
        if self.cu_seqlens is not None:
            cu = self.cu_seqlens.to(device) if device is not None else self.cu_seqlens
            kw.update(cu_seqlens_q=cu, cu_seqlens_k=cu, max_seqlen_q=self.max_seqlen,
                      max_seqlen_k=self.max_seqlen)
        return kw

    def oracle_mask_kwargs(self) -> dict:
        """The same variant in the CPU oracle's vocabulary: one segment id per
        key position (largest k with start_k <= position, -1 before the first
        start) and the global positions as a list."""
        wl = self.wl
        kw = dict(prefix_len=wl.prefix_len, relpos=wl.relpos, norm=NORM_CODES[wl.norm],
                  query_start=wl.query_start)
        if wl.mask == MASK_GLOBAL_WINDOW:
            kw["global_tokens"] = list(wl.global_list) if wl.global_list else \
                list(range(wl.num_global))
        if self.segment_starts is not None:
            S = self.max_seqlen
            ids = [-1] * S
            for k, st in enumerate(self.segment_starts.tolist()):
                for pos in range(st, S):
                    ids[pos] = k
            kw["token_ids"] = ids
        return kw


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
    seg = None
    if wl.mask in (MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE):
        S = max(lengths) if wl.varlen else wl.seqlen
        lo = wl.prefix_len if wl.mask == MASK_SHARE_QUESTION else 0
        hi = S if wl.mask == MASK_SHARE_QUESTION else min(wl.query_start, S)
        n = max(1, min(wl.num_segments, hi - lo))
        cuts = (torch.randperm(max(hi - lo - 1, 0), generator=g)[:n - 1] + lo + 1).tolist()
        seg = torch.tensor(sorted([lo] + cuts), dtype=torch.int32)
    return Inputs(wl, q, k, v, slopes, cu, lengths, seg)

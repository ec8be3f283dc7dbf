"""MI355X (gfx950) fused attention forward.

`fwd` marshals torch tensors (device memory and the current stream) into an
`attn_variant_desc` and calls `attn_fwd` of libattn.so. The computation runs
entirely in the library's HIP kernels; if the library is missing the import
of `fwd`'s backend fails loudly.

The C ABI sees only pointers, so every shape is checked here against q before
the call: a mismatch raises ValueError (TypeError for a dtype or device) and
nothing is launched.
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional

import torch

from ._abi import (ATTN_BF16, ATTN_FLAG_LOG, ATTN_FLAG_VALIDATE, ATTN_FP32, ATTN_MASK_CAUSAL,  # noqa: F401
                   ATTN_MASK_CAUSAL_BLOCKWISE, ATTN_MASK_GLOBAL_SLIDING_WINDOW, ATTN_MASK_NONE,
                   ATTN_MASK_PREFIX_LM, ATTN_MASK_SHARE_QUESTION, ATTN_MASK_SLIDING_WINDOW,
                   ATTN_MAX_SEGMENTS, ATTN_NORM_RELU, ATTN_NORM_SIGMOID, ATTN_NORM_SOFTMAX,
                   AttnError, AttnVariantDesc, check, load, plan_tiles, row_range)

__all__ = ["fwd", "make_desc", "lse_shape", "AttnError", "AttnVariantDesc", "load", "plan_tiles",
           "row_range", "ATTN_BF16", "ATTN_FP32", "ATTN_MASK_NONE", "ATTN_MASK_CAUSAL",
           "ATTN_MASK_SLIDING_WINDOW", "ATTN_MASK_PREFIX_LM", "ATTN_MASK_GLOBAL_SLIDING_WINDOW",
           "ATTN_MASK_SHARE_QUESTION", "ATTN_MASK_CAUSAL_BLOCKWISE", "ATTN_NORM_SOFTMAX",
           "ATTN_NORM_RELU", "ATTN_NORM_SIGMOID", "ATTN_FLAG_VALIDATE", "ATTN_FLAG_LOG"]

_DTYPES = {torch.bfloat16: ATTN_BF16, torch.float32: ATTN_FP32}
_MASKS = {"none": ATTN_MASK_NONE, "causal": ATTN_MASK_CAUSAL,
          "sliding_window": ATTN_MASK_SLIDING_WINDOW, "prefix_lm": ATTN_MASK_PREFIX_LM,
          "global_sliding_window": ATTN_MASK_GLOBAL_SLIDING_WINDOW,
          "share_question": ATTN_MASK_SHARE_QUESTION,
          "causal_blockwise": ATTN_MASK_CAUSAL_BLOCKWISE}
_NORMS = {"softmax": ATTN_NORM_SOFTMAX, "relu": ATTN_NORM_RELU, "sigmoid": ATTN_NORM_SIGMOID}
_ORDERS = {None: 0, "natural": 1, "xcd_groups": 2}


def _int_array(t, name, device):
    if t.dtype != torch.int32 or t.device != device or not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous int32 on q's device")
    if t.dim() != 1:
        raise ValueError(f"{name} must be one-dimensional")


def _layout_array(t, name, device, nseq):
    """An index-mask layout: one int32 array shared by every sequence, or one
    row per sequence ([nseq, n], rows contiguous). Returns (entries, stride)."""
    if t.dtype != torch.int32 or t.device != device:
        raise TypeError(f"{name} must be int32 on q's device")
    if t.dim() == 1:
        if not t.is_contiguous():
            raise TypeError(f"{name} must be contiguous")
        return t.numel(), 0
    if t.dim() != 2 or t.shape[0] != nseq:
        raise ValueError(f"{name} must be [n] or [{nseq} sequences, n], got {tuple(t.shape)}")
    if t.shape[1] > 0 and (t.stride(1) != 1 or t.stride(0) < t.shape[1]):
        raise ValueError(f"{name} rows must be contiguous and not overlap")
    return t.shape[1], t.stride(0) if t.shape[1] > 0 else 0


def lse_shape(q, varlen: bool):
    """Shape of the fp32 LSE output for q: (B, Hq, Sq), or (Hq, Tq) when varlen."""
    return (q.shape[1], q.shape[0]) if varlen else (q.shape[0], q.shape[1], q.shape[2])


def _check_shapes(q, k, v, out, varlen, alibi_slopes):
    want = 3 if varlen else 4
    layout = "[T, H, D]" if varlen else "[B, H, S, D]"
    for name, t in (("q", q), ("k", k), ("v", v), ("out", out)):
        if t.dim() != want:
            raise ValueError(f"{name} must be {layout}, got shape {tuple(t.shape)}")
        if t.device != q.device:
            raise TypeError(f"{name} is on {t.device}, q on {q.device}")
        if t.stride(-1) != 1:
            raise ValueError("head_dim must be the innermost, contiguous axis")
    if k.shape != v.shape:
        raise ValueError(f"k {tuple(k.shape)} and v {tuple(v.shape)} differ")
    if k.shape[-1] != q.shape[-1]:
        raise ValueError(f"head_dim of k ({k.shape[-1]}) differs from q ({q.shape[-1]})")
    if out.shape != q.shape:
        raise ValueError(f"out {tuple(out.shape)} must have q's shape {tuple(q.shape)}")
    if not varlen and k.shape[0] != q.shape[0]:
        raise ValueError(f"batch of k/v ({k.shape[0]}) differs from q ({q.shape[0]})")
    if alibi_slopes is not None:
        if alibi_slopes.dtype != torch.float32 or alibi_slopes.device != q.device \
                or not alibi_slopes.is_contiguous():
            raise TypeError("alibi_slopes must be contiguous fp32 on q's device")
        hq = q.shape[1]
        if alibi_slopes.numel() != hq:
            raise ValueError(f"alibi_slopes has {alibi_slopes.numel()} entries, q has {hq} heads")


def make_desc(q, k, v, out, *, causal=False, window=None, alibi_slopes=None, softcap=0.0,
              scale=None, cu_seqlens_q=None, cu_seqlens_k=None, max_seqlen_q=None,
              max_seqlen_k=None, stream=None, mask=None, prefix_len=0, num_global=0,
              global_tokens=None, segment_starts=None, query_start=0, relative_position=False,
              norm="softmax", validate=False, heads_per_wg=0, order=None,
              chunk=0, log=False) -> AttnVariantDesc:
    """Build the descriptor for tensors q/k/v/out (see include/attn.h for layouts).

    `mask` names any attn_mask_kind_t ("prefix_lm", "global_sliding_window",
    "share_question", "causal_blockwise", ...) and overrides causal/window;
    `window` gives the (left, right) bounds of the two window masks;
    `global_tokens` (device int32, strictly increasing) lists the global
    positions of the global sliding window (else positions 0..num_global-1).
    `segment_starts` and `global_tokens` are one array shared by every
    sequence, or one row per sequence ([batch, n]; per-sequence layouts).
    `validate` sets ATTN_FLAG_VALIDATE (host check of cu_seqlens, segments and
    global positions), `log` ATTN_FLAG_LOG (the launch plan on stderr). `heads_per_wg`, `order` ("natural", "xcd_groups") and
    `chunk` override the library's workgroup schedule (tuning and tests).
    """
    if q.dtype not in _DTYPES or k.dtype != q.dtype or v.dtype != q.dtype or out.dtype != q.dtype:
        raise TypeError("q, k, v, out must share dtype bfloat16 or float32")
    varlen = cu_seqlens_q is not None
    _check_shapes(q, k, v, out, varlen, alibi_slopes)
    d = AttnVariantDesc.new()
    d.dtype = _DTYPES[q.dtype]
    D = q.shape[-1]
    d.head_dim = D
    d.scale = float(scale) if scale is not None else 1.0 / math.sqrt(D)
    if mask is not None:
        d.mask_kind = _MASKS[mask] if isinstance(mask, str) else int(mask)
    elif window is not None:
        d.mask_kind = ATTN_MASK_SLIDING_WINDOW
    else:
        d.mask_kind = ATTN_MASK_CAUSAL if causal else ATTN_MASK_NONE
    if window is not None:
        d.window_left, d.window_right = int(window[0]), int(window[1])
    else:
        d.window_left = d.window_right = -1
    d.prefix_len, d.num_global, d.query_start = int(prefix_len), int(num_global), int(query_start)
    d.relative_position = 1 if relative_position else 0
    d.norm_kind = _NORMS[norm] if isinstance(norm, str) else int(norm)
    nseq = (cu_seqlens_q.numel() - 1) if varlen else q.shape[0]
    if segment_starts is not None:
        d.num_segments, d.segment_stride = _layout_array(segment_starts, "segment_starts",
                                                         q.device, nseq)
        d.segment_starts = segment_starts.data_ptr()
    if global_tokens is not None:
        n, d.global_stride = _layout_array(global_tokens, "global_tokens", q.device, nseq)
        if num_global and int(num_global) != n:
            raise ValueError(f"num_global={num_global} but global_tokens has {n} entries")
        d.num_global = n
        d.global_tokens = global_tokens.data_ptr() if n else None
    d.softcap = float(softcap)
    if alibi_slopes is not None:
        d.alibi_slopes = alibi_slopes.data_ptr()
    if varlen:
        if cu_seqlens_k is None:
            cu_seqlens_k = cu_seqlens_q
        _int_array(cu_seqlens_q, "cu_seqlens_q", q.device)
        _int_array(cu_seqlens_k, "cu_seqlens_k", q.device)
        if cu_seqlens_k.numel() != cu_seqlens_q.numel() or cu_seqlens_q.numel() < 1:
            raise ValueError(f"cu_seqlens_q ({cu_seqlens_q.numel()}) and cu_seqlens_k "
                             f"({cu_seqlens_k.numel()}) must both hold batch + 1 >= 1 entries")
        if max_seqlen_q is None or max_seqlen_k is None:
            raise ValueError("varlen needs max_seqlen_q and max_seqlen_k (no device readback)")
        d.batch = cu_seqlens_q.numel() - 1
        d.num_q_heads, d.num_kv_heads = q.shape[1], k.shape[1]
        d.cu_seqlens_q, d.cu_seqlens_k = cu_seqlens_q.data_ptr(), cu_seqlens_k.data_ptr()
        d.max_seqlen_q, d.max_seqlen_k = int(max_seqlen_q), int(max_seqlen_k)
        d.total_q, d.total_k = q.shape[0], k.shape[0]
        for name, t in (("q", q), ("k", k), ("v", v), ("o", out)):
            setattr(d, f"stride_{name}_h", t.stride(1))
            setattr(d, f"stride_{name}_s", t.stride(0))
    else:
        d.batch, d.num_q_heads, d.seqlen_q = q.shape[0], q.shape[1], q.shape[2]
        d.num_kv_heads, d.seqlen_k = k.shape[1], k.shape[2]
        for name, t in (("q", q), ("k", k), ("v", v), ("o", out)):
            setattr(d, f"stride_{name}_b", t.stride(0))
            setattr(d, f"stride_{name}_h", t.stride(1))
            setattr(d, f"stride_{name}_s", t.stride(2))
    d.flags = (ATTN_FLAG_VALIDATE if validate else 0) | (ATTN_FLAG_LOG if log else 0)
    d.sched_heads_per_wg = int(heads_per_wg)
    d.sched_order = _ORDERS[order]
    d.sched_chunk = int(chunk)
    if stream is None:
        stream = torch.cuda.current_stream(q.device).cuda_stream
    d.stream = stream
    return d


def fwd(q, k, v, *, causal: bool = False, window=None, alibi_slopes=None, softcap: float = 0.0,
        scale: Optional[float] = None, cu_seqlens_q=None, cu_seqlens_k=None, max_seqlen_q=None,
        max_seqlen_k=None, out=None, lse=None, return_lse: bool = True, mask=None,
        prefix_len: int = 0, num_global: int = 0, global_tokens=None, segment_starts=None,
        query_start: int = 0, relative_position: bool = False, norm="softmax",
        validate: bool = False, heads_per_wg: int = 0, order=None, chunk: int = 0,
        log: bool = False):
    """Attention forward on the GPU.

    Fixed length: q [B,Hq,S,D], k/v [B,Hkv,Sk,D] -> out like q, lse [B,Hq,S] fp32.
    Varlen: q [Tq,Hq,D], k/v [Tk,Hkv,D], cu_seqlens int32 [B+1] -> lse [Hq,Tq].
    window=(left, right) selects the sliding-window mask (-1 = unbounded).
    The other variants of include/attn.h are selected by `mask` (with
    prefix_len, num_global / global_tokens, segment_starts, query_start),
    `relative_position` and `norm` ("softmax", "relu", "sigmoid"; only softmax
    produces an LSE). See make_desc for `validate` and the schedule overrides.
    """
    if not q.is_cuda:
        raise ValueError("fwd runs on the GPU only; q, k, v must be device tensors")
    lib = load()
    varlen = cu_seqlens_q is not None
    if out is None:
        out = torch.empty_like(q)
    softmax = (_NORMS[norm] if isinstance(norm, str) else int(norm)) == ATTN_NORM_SOFTMAX
    if not softmax:
        return_lse, lse = False, None
    if lse is None and return_lse:
        lse = torch.empty(lse_shape(q, varlen), dtype=torch.float32, device=q.device)
    if lse is not None:
        if lse.dtype != torch.float32 or not lse.is_contiguous() or lse.device != q.device:
            raise TypeError("lse must be contiguous fp32 on q's device")
        if tuple(lse.shape) != tuple(lse_shape(q, varlen)):
            raise ValueError(f"lse {tuple(lse.shape)} must be {tuple(lse_shape(q, varlen))}")
    d = make_desc(q, k, v, out, causal=causal, window=window, alibi_slopes=alibi_slopes,
                  softcap=softcap, scale=scale, cu_seqlens_q=cu_seqlens_q,
                  cu_seqlens_k=cu_seqlens_k, max_seqlen_q=max_seqlen_q,
                  max_seqlen_k=max_seqlen_k, mask=mask, prefix_len=prefix_len,
                  num_global=num_global, global_tokens=global_tokens,
                  segment_starts=segment_starts, query_start=query_start,
                  relative_position=relative_position, norm=norm, validate=validate,
                  heads_per_wg=heads_per_wg, order=order, chunk=chunk, log=log)
    status = lib.attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                          lse.data_ptr() if lse is not None else None, ctypes.byref(d))
    check(status, lib)
    return (out, lse) if return_lse else out

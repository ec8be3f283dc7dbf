"""CPU oracle for the attention forward pass (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product library never loads it and shares no code
with it. The arithmetic lives in `attn_ref.c` (plain C, fp64, materialised
scores); this module builds it with gcc and marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "attn_ref.c")
_LIB = os.path.join(_HERE, "libattn_ref.so")

MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW = 0, 1, 2
MASK_PREFIX_LM, MASK_GLOBAL_WINDOW, MASK_SHARE_QUESTION, MASK_CAUSAL_BLOCKWISE = 3, 4, 5, 6
NORM_SOFTMAX, NORM_RELU, NORM_SIGMOID = 0, 1, 2


class _RefParams(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("hq", ctypes.c_int32),
        ("hkv", ctypes.c_int32),
        ("sq", ctypes.c_int32),
        ("sk", ctypes.c_int32),
        ("d", ctypes.c_int32),
        ("scale", ctypes.c_double),
        ("mask_kind", ctypes.c_int32),
        ("window_left", ctypes.c_int32),
        ("window_right", ctypes.c_int32),
        ("slopes", ctypes.POINTER(ctypes.c_double)),
        ("softcap", ctypes.c_double),
        ("cu_q", ctypes.POINTER(ctypes.c_int32)),
        ("cu_k", ctypes.POINTER(ctypes.c_int32)),
        ("prefix_len", ctypes.c_int32),
        ("relpos", ctypes.c_int32),
        ("norm_kind", ctypes.c_int32),
        ("token_ids", ctypes.POINTER(ctypes.c_int32)),
        ("query_start", ctypes.c_int32),
        ("global_tokens", ctypes.POINTER(ctypes.c_int32)),
        ("num_global", ctypes.c_int32),
    ]


def build(src: str = _SRC, out: str = _LIB, extra_flags: Sequence[str] = ()) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, strict IEEE: no fast-math)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           "-fno-fast-math", *extra_flags, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _stale() -> bool:
    return (not os.path.exists(_LIB)) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)


_lib = None


def load(path: Optional[str] = None):
    """Load (building first if missing or older than its source) the oracle."""
    global _lib
    if path is not None:
        lib = ctypes.CDLL(path)
    else:
        if _lib is not None:
            return _lib
        if _stale():
            build()
        lib = ctypes.CDLL(_LIB)
    lib.attn_ref_fwd.restype = ctypes.c_int
    lib.attn_ref_fwd.argtypes = [ctypes.POINTER(_RefParams)] + [ctypes.c_void_p] * 5 + [
        ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.attn_ref_num_threads.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def num_threads() -> int:
    return int(load().attn_ref_num_threads())


def _f32(x) -> np.ndarray:
    """Exact fp32 copy of a torch tensor (bf16 and fp32 values are exact in fp32)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return np.ascontiguousarray(x.detach().to("cpu", torch.float32).numpy())
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(x, dtype=np.float32))


def _i32(x) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return np.ascontiguousarray(x.detach().to("cpu", torch.int32).numpy())
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def attention(q, k, v, *, scale: float, mask: int = MASK_NONE, window_left: int = -1,
              window_right: int = -1, slopes=None, softcap: float = 0.0,
              cu_seqlens_q=None, cu_seqlens_k=None, rows=None, want_probs: bool = False,
              prefix_len: int = 0, relpos: bool = False, norm: int = NORM_SOFTMAX,
              token_ids=None, query_start: int = 0, global_tokens=None, lib=None):
    """Reference attention forward.

    Fixed length: q [B,Hq,Sq,D], k/v [B,Hkv,Sk,D] -> o [B,Hq,Sq,D], lse [B,Hq,Sq].
    Varlen (cu_seqlens given): q [Tq,Hq,D], k/v [Tk,Hkv,D] -> o [Tq,Hq,D], lse [Hq,Tq].
    `rows`: optional flat LSE indices to compute; other rows are left NaN.
    PrefixLM uses `prefix_len`; the share-question and causal-blockwise masks
    use `token_ids` (one id per key position; blockwise also `query_start`);
    the global sliding window uses the window bounds and `global_tokens`.
    `norm` selects softmax, ReLU(S)/L or Sigmoid(S)/L (the last two have no
    LSE: NaN). Returns (o, lse) as float64 numpy arrays, plus P [B,Hq,Sq,Sk]
    if want_probs.
    """
    lib = lib or load()
    qn, kn, vn = _f32(q), _f32(k), _f32(v)
    varlen = cu_seqlens_q is not None
    p = _RefParams()
    if varlen:
        cuq = _i32(cu_seqlens_q)
        cuk = _i32(cu_seqlens_k if cu_seqlens_k is not None else cu_seqlens_q)
        tq, hq, d = qn.shape
        hkv = kn.shape[1]
        p.batch, p.hq, p.hkv, p.sq, p.sk, p.d = len(cuq) - 1, hq, hkv, 0, 0, d
        p.cu_q = cuq.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        p.cu_k = cuk.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        lse_shape = (hq, tq)
    else:
        b, hq, sq, d = qn.shape
        hkv, sk = kn.shape[1], kn.shape[2]
        p.batch, p.hq, p.hkv, p.sq, p.sk, p.d = b, hq, hkv, sq, sk, d
        lse_shape = (b, hq, sq)
    p.scale = float(scale)
    p.mask_kind = int(mask)
    p.window_left, p.window_right = int(window_left), int(window_right)
    p.softcap = float(softcap)
    p.prefix_len = int(prefix_len)
    p.relpos = 1 if relpos else 0
    p.norm_kind = int(norm)
    p.query_start = int(query_start)
    ids = None
    if token_ids is not None:
        ids = _i32(token_ids)
        p.token_ids = ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    gl = None
    if global_tokens is not None:
        gl = _i32(global_tokens)
        p.global_tokens = gl.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        p.num_global = int(gl.size)
    sl = None
    if slopes is not None:
        sl = np.ascontiguousarray(np.asarray(_f32(slopes), dtype=np.float64))
        p.slopes = sl.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    o = np.full(qn.shape, np.nan, dtype=np.float64)
    lse = np.full(lse_shape, np.nan, dtype=np.float64)
    rows_arr = None
    nrows = 0
    if rows is not None:
        rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        nrows = rows_arr.size
    probs = None
    if want_probs:
        if varlen:
            raise ValueError("probs are only produced for fixed-length inputs")
        probs = np.zeros((p.batch, p.hq, p.sq, p.sk), dtype=np.float64)
    rc = lib.attn_ref_fwd(ctypes.byref(p), qn.ctypes.data, kn.ctypes.data, vn.ctypes.data,
                          o.ctypes.data, lse.ctypes.data,
                          rows_arr.ctypes.data if rows_arr is not None else None, nrows,
                          probs.ctypes.data if probs is not None else None)
    if rc != 0:
        raise ValueError("oracle rejected its parameters")
    del sl, ids, gl
    if want_probs:
        return o, lse, probs
    return o, lse


def attention_inputs(inp, rows=None, **kw):
    """Run the oracle on a `workloads.Inputs` bundle."""
    wl = inp.wl
    return attention(inp.q, inp.k, inp.v, scale=wl.scale, mask=wl.mask,
                     window_left=wl.window_left, window_right=wl.window_right,
                     slopes=inp.slopes, softcap=wl.softcap,
                     cu_seqlens_q=inp.cu_seqlens, cu_seqlens_k=inp.cu_seqlens,
                     rows=rows, **{**inp.oracle_mask_kwargs(), **kw})

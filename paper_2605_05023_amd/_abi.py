"""ctypes mirror of include/attn.h and the loader of libattn.so.

Argument marshalling only: every step of the computation runs in the HIP
kernels of libattn.so. There is no fallback; loading fails loudly when the
library has not been built.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libattn.so")

ATTN_ABI_VERSION = 4
ATTN_MAX_SEGMENTS = 2048
ATTN_FLAG_VALIDATE = 1
ATTN_FLAG_LOG = 2
ATTN_BF16, ATTN_FP32 = 0, 1
ATTN_MASK_NONE, ATTN_MASK_CAUSAL, ATTN_MASK_SLIDING_WINDOW = 0, 1, 2
ATTN_MASK_PREFIX_LM, ATTN_MASK_GLOBAL_SLIDING_WINDOW = 3, 4
ATTN_MASK_SHARE_QUESTION, ATTN_MASK_CAUSAL_BLOCKWISE = 5, 6
ATTN_NORM_SOFTMAX, ATTN_NORM_RELU, ATTN_NORM_SIGMOID = 0, 1, 2

STATUS = {
    0: "ATTN_OK",
    -1: "ATTN_ERR_NULL_PTR",
    -2: "ATTN_ERR_BAD_SHAPE",
    -3: "ATTN_ERR_BAD_VARIANT",
    -4: "ATTN_ERR_ALIGNMENT",
    -5: "ATTN_ERR_UNSUPPORTED",
    -6: "ATTN_ERR_ABI",
    -7: "ATTN_ERR_LAUNCH",
}
STATUS_CODE = {v: k for k, v in STATUS.items()}

EXPORTED = ("attn_fwd", "attn_status_string", "attn_abi_version", "attn_plan_tiles",
            "attn_row_range")


class AttnVariantDesc(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("dtype", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("seqlen_q", ctypes.c_int32),
        ("seqlen_k", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("mask_kind", ctypes.c_int32),
        ("window_left", ctypes.c_int32),
        ("window_right", ctypes.c_int32),
        ("alibi_slopes", ctypes.c_void_p),
        ("softcap", ctypes.c_float),
        ("cu_seqlens_q", ctypes.c_void_p),
        ("cu_seqlens_k", ctypes.c_void_p),
        ("max_seqlen_q", ctypes.c_int32),
        ("max_seqlen_k", ctypes.c_int32),
        ("total_q", ctypes.c_int64),
        ("total_k", ctypes.c_int64),
        ("stride_q_b", ctypes.c_int64), ("stride_q_h", ctypes.c_int64), ("stride_q_s", ctypes.c_int64),
        ("stride_k_b", ctypes.c_int64), ("stride_k_h", ctypes.c_int64), ("stride_k_s", ctypes.c_int64),
        ("stride_v_b", ctypes.c_int64), ("stride_v_h", ctypes.c_int64), ("stride_v_s", ctypes.c_int64),
        ("stride_o_b", ctypes.c_int64), ("stride_o_h", ctypes.c_int64), ("stride_o_s", ctypes.c_int64),
        ("stream", ctypes.c_void_p),
        ("norm_kind", ctypes.c_int32),
        ("relative_position", ctypes.c_int32),
        ("prefix_len", ctypes.c_int32),
        ("num_global", ctypes.c_int32),
        ("segment_starts", ctypes.c_void_p),
        ("num_segments", ctypes.c_int32),
        ("query_start", ctypes.c_int32),
        ("global_tokens", ctypes.c_void_p),
        ("flags", ctypes.c_uint32),
        ("sched_heads_per_wg", ctypes.c_int32),
        ("sched_order", ctypes.c_int32),
        ("sched_chunk", ctypes.c_int32),
        ("segment_stride", ctypes.c_int64),
        ("global_stride", ctypes.c_int64),
    ]

    @classmethod
    def new(cls) -> "AttnVariantDesc":
        d = cls()
        d.struct_size = ctypes.sizeof(cls)
        return d


class AttnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH):
    """Load libattn.so; raise if it is missing (build it with
    `python -m paper_2605_05023_amd.build`)."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2605_05023_amd.build`")
    lib = ctypes.CDLL(path)
    lib.attn_fwd.restype = ctypes.c_int
    lib.attn_fwd.argtypes = [ctypes.c_void_p] * 5 + [ctypes.POINTER(AttnVariantDesc)]
    lib.attn_status_string.restype = ctypes.c_char_p
    lib.attn_status_string.argtypes = [ctypes.c_int]
    lib.attn_abi_version.restype = ctypes.c_int
    lib.attn_abi_version.argtypes = []
    lib.attn_plan_tiles.restype = ctypes.c_int
    lib.attn_plan_tiles.argtypes = [ctypes.POINTER(AttnVariantDesc), ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.POINTER(ctypes.c_int32)]
    lib.attn_row_range.restype = ctypes.c_int
    lib.attn_row_range.argtypes = [ctypes.POINTER(AttnVariantDesc), ctypes.POINTER(ctypes.c_int32),
                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.POINTER(ctypes.c_int32)]
    if lib.attn_abi_version() != ATTN_ABI_VERSION:
        raise ImportError("libattn.so ABI version mismatch")
    if path == LIB_PATH:
        _lib = lib
    return lib


def check(status: int, lib=None) -> None:
    if status != 0:
        lib = lib or load()
        raise AttnError(status, lib.attn_status_string(status).decode())


def plan_tiles(mask_kind: int, window_left: int, window_right: int, q0: int, rows: int, lq: int,
               lk: int, block_n: int, lib=None, prefix_len: int = 0):
    """Host mirror of the in-kernel tile planner: (lo, full_lo, full_hi, hi)."""
    lib = lib or load()
    d = AttnVariantDesc.new()
    d.mask_kind, d.window_left, d.window_right = mask_kind, window_left, window_right
    d.prefix_len = prefix_len
    d.scale = 1.0
    out = (ctypes.c_int32 * 4)()
    check(lib.attn_plan_tiles(ctypes.byref(d), q0, rows, lq, lk, block_n, out), lib)
    return tuple(out)


def row_range(desc: AttnVariantDesc, i: int, lq: int, lk: int, segment_starts=None, lib=None):
    """Host mirror of the kernels' per-row visibility: (pfx, jlo, jhi), keys
    j < pfx and jlo <= j <= jhi are visible. `segment_starts`: host ints."""
    lib = lib or load()
    seg = None
    if segment_starts is not None:
        seg = (ctypes.c_int32 * max(1, len(segment_starts)))(*segment_starts)
    out = (ctypes.c_int32 * 3)()
    check(lib.attn_row_range(ctypes.byref(desc), seg, i, lq, lk, out), lib)
    return tuple(out)

"""The C ABI of libattn.so on the CPU: symbols, versions and every validation
error path. Validation runs before any HIP call, so none of these calls
touches a GPU (pointers are dummies that are never dereferenced)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2605_05023_amd as attn
from paper_2605_05023_amd import _abi

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "attn.h")
P = 0x10000  # dummy 16-byte aligned device pointers, never dereferenced


@pytest.fixture(scope="module")
def lib():
    return attn.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(attn_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(_abi.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_ctypes_mirror_matches_header(tmp_path):
    """Compile the header with gcc and compare sizeof and every field offset."""
    fields = [f[0] for f in _abi.AttnVariantDesc._fields_]
    src = tmp_path / "layout.c"
    lines = ["#include <stdio.h>", "#include <stddef.h>", f'#include "{HEADER}"', "int main(void) {",
             '  printf("%zu\\n", sizeof(attn_variant_desc));']
    lines += [f'  printf("%zu\\n", offsetof(attn_variant_desc, {f}));' for f in fields]
    lines += ["  return 0;", "}"]
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", str(src), "-o", str(exe)], check=True)
    out = [int(x) for x in subprocess.run([str(exe)], check=True, capture_output=True,
                                          text=True).stdout.split()]
    assert out[0] == ctypes.sizeof(_abi.AttnVariantDesc)
    for f, off in zip(fields, out[1:]):
        assert getattr(_abi.AttnVariantDesc, f).offset == off, f


def test_versions_and_strings(lib):
    assert lib.attn_abi_version() == _abi.ATTN_ABI_VERSION
    for code in _abi.STATUS:
        s = lib.attn_status_string(code)
        assert s and s != b"unknown status"
    assert lib.attn_status_string(-99) == b"unknown status"


def base_desc(varlen=False):
    d = _abi.AttnVariantDesc.new()
    d.dtype = _abi.ATTN_BF16
    d.batch, d.num_q_heads, d.num_kv_heads = 2, 8, 2
    d.head_dim = 128
    d.scale = 0.125
    d.mask_kind = _abi.ATTN_MASK_CAUSAL
    if varlen:
        d.cu_seqlens_q = d.cu_seqlens_k = P
        d.max_seqlen_q = d.max_seqlen_k = 100
        d.total_q = d.total_k = 150
    else:
        d.seqlen_q = d.seqlen_k = 100
    return d


def call(lib, d, q=P, k=P, v=P, o=P, lse=P):
    return lib.attn_fwd(q, k, v, o, lse, ctypes.byref(d) if d is not None else None)


def err(name):
    return _abi.STATUS_CODE[name]


CASES = [
    ("struct_size", lambda d: setattr(d, "struct_size", 8), "ATTN_ERR_ABI"),
    ("dtype", lambda d: setattr(d, "dtype", 7), "ATTN_ERR_UNSUPPORTED"),
    ("head_dim 96", lambda d: setattr(d, "head_dim", 96), "ATTN_ERR_UNSUPPORTED"),
    ("head_dim 0", lambda d: setattr(d, "head_dim", 0), "ATTN_ERR_UNSUPPORTED"),
    ("gqa ratio", lambda d: setattr(d, "num_kv_heads", 3), "ATTN_ERR_BAD_SHAPE"),
    ("zero q heads", lambda d: setattr(d, "num_q_heads", 0), "ATTN_ERR_BAD_SHAPE"),
    ("zero kv heads", lambda d: setattr(d, "num_kv_heads", 0), "ATTN_ERR_BAD_SHAPE"),
    ("negative batch", lambda d: setattr(d, "batch", -1), "ATTN_ERR_BAD_SHAPE"),
    ("negative seqlen", lambda d: setattr(d, "seqlen_q", -5), "ATTN_ERR_BAD_SHAPE"),
    ("mask kind", lambda d: setattr(d, "mask_kind", 9), "ATTN_ERR_BAD_VARIANT"),
    ("window < -1", lambda d: (setattr(d, "mask_kind", 2), setattr(d, "window_left", -2)),
     "ATTN_ERR_BAD_VARIANT"),
    ("window right < -1", lambda d: (setattr(d, "mask_kind", 2), setattr(d, "window_right", -7)),
     "ATTN_ERR_BAD_VARIANT"),
    ("softcap < 0", lambda d: setattr(d, "softcap", -1.0), "ATTN_ERR_BAD_VARIANT"),
    ("softcap nan", lambda d: setattr(d, "softcap", float("nan")), "ATTN_ERR_BAD_VARIANT"),
    ("scale 0", lambda d: setattr(d, "scale", 0.0), "ATTN_ERR_BAD_VARIANT"),
    ("scale < 0", lambda d: setattr(d, "scale", -0.1), "ATTN_ERR_BAD_VARIANT"),
    ("scale inf", lambda d: setattr(d, "scale", float("inf")), "ATTN_ERR_BAD_VARIANT"),
    ("stride not 16B", lambda d: setattr(d, "stride_q_s", 132), "ATTN_ERR_ALIGNMENT"),
    ("head stride not 16B", lambda d: setattr(d, "stride_k_h", 100 * 128 + 4), "ATTN_ERR_ALIGNMENT"),
    ("rows overlap", lambda d: setattr(d, "stride_v_s", 64), "ATTN_ERR_BAD_SHAPE"),
    ("negative stride", lambda d: setattr(d, "stride_o_h", -128), "ATTN_ERR_BAD_SHAPE"),
    ("slice beyond 2 GiB", lambda d: (setattr(d, "seqlen_k", 1 << 20), setattr(d, "stride_k_s", 1 << 12)),
     "ATTN_ERR_UNSUPPORTED"),
    # one key row past the largest slice the 32-bit offsets allow (with one
    # tile of padding): ((Sk + 128) * 128 + 128) * 2 bytes reaches 2^31
    ("slice one row past 2 GiB", lambda d: (setattr(d, "batch", 1), setattr(d, "num_q_heads", 1),
                                            setattr(d, "num_kv_heads", 1),
                                            setattr(d, "seqlen_k", (1 << 23) - 129)),
     "ATTN_ERR_UNSUPPORTED"),
    ("cu_k without cu_q", lambda d: setattr(d, "cu_seqlens_k", P), "ATTN_ERR_BAD_SHAPE"),
    ("grid beyond int32", lambda d: (setattr(d, "batch", 1 << 21), setattr(d, "num_q_heads", 1 << 10),
                                     setattr(d, "num_kv_heads", 1 << 10), setattr(d, "seqlen_q", 1),
                                     setattr(d, "seqlen_k", 1)), "ATTN_ERR_UNSUPPORTED"),
    ("mask kind 7", lambda d: setattr(d, "mask_kind", 7), "ATTN_ERR_BAD_VARIANT"),
    ("mask kind < 0", lambda d: setattr(d, "mask_kind", -1), "ATTN_ERR_BAD_VARIANT"),
    ("norm kind 3", lambda d: setattr(d, "norm_kind", 3), "ATTN_ERR_BAD_VARIANT"),
    ("norm kind < 0", lambda d: setattr(d, "norm_kind", -1), "ATTN_ERR_BAD_VARIANT"),
    ("relative_position 2", lambda d: setattr(d, "relative_position", 2), "ATTN_ERR_BAD_VARIANT"),
    ("prefix < 0", lambda d: (setattr(d, "mask_kind", 3), setattr(d, "prefix_len", -1)),
     "ATTN_ERR_BAD_VARIANT"),
    ("global window < -1", lambda d: (setattr(d, "mask_kind", 4), setattr(d, "window_left", -3)),
     "ATTN_ERR_BAD_VARIANT"),
    ("num_global < 0", lambda d: (setattr(d, "mask_kind", 4), setattr(d, "num_global", -1)),
     "ATTN_ERR_BAD_VARIANT"),
    ("no segments", lambda d: (setattr(d, "mask_kind", 5), setattr(d, "segment_starts", P),
                               setattr(d, "num_segments", 0)), "ATTN_ERR_BAD_VARIANT"),
    ("too many segments", lambda d: (setattr(d, "mask_kind", 6), setattr(d, "segment_starts", P),
                                     setattr(d, "num_segments", _abi.ATTN_MAX_SEGMENTS + 1)),
     "ATTN_ERR_BAD_VARIANT"),
    ("query_start < 0", lambda d: (setattr(d, "mask_kind", 6), setattr(d, "segment_starts", P),
                                   setattr(d, "num_segments", 2), setattr(d, "query_start", -4)),
     "ATTN_ERR_BAD_VARIANT"),
    ("segments missing", lambda d: (setattr(d, "mask_kind", 5), setattr(d, "num_segments", 3)),
     "ATTN_ERR_NULL_PTR"),
    # 2 log2(e) scale / C overflows fp32 for a tiny cap
    ("softcap too small", lambda d: setattr(d, "softcap", 1e-40), "ATTN_ERR_BAD_VARIANT"),
    ("too many global positions", lambda d: (setattr(d, "mask_kind", 4), setattr(d, "global_tokens", P),
                                             setattr(d, "num_global", _abi.ATTN_MAX_SEGMENTS + 1)),
     "ATTN_ERR_BAD_VARIANT"),
    ("unknown flag", lambda d: setattr(d, "flags", 4), "ATTN_ERR_BAD_VARIANT"),
    ("negative segment stride", lambda d: (setattr(d, "mask_kind", 5), setattr(d, "segment_starts", P),
                                           setattr(d, "num_segments", 3),
                                           setattr(d, "segment_stride", -3)), "ATTN_ERR_BAD_VARIANT"),
    ("segment rows overlap", lambda d: (setattr(d, "mask_kind", 6), setattr(d, "segment_starts", P),
                                        setattr(d, "num_segments", 3),
                                        setattr(d, "segment_stride", 2)), "ATTN_ERR_BAD_VARIANT"),
    ("negative global stride", lambda d: (setattr(d, "mask_kind", 4), setattr(d, "global_tokens", P),
                                          setattr(d, "num_global", 3),
                                          setattr(d, "global_stride", -1)), "ATTN_ERR_BAD_VARIANT"),
    ("global rows overlap", lambda d: (setattr(d, "mask_kind", 4), setattr(d, "global_tokens", P),
                                       setattr(d, "num_global", 3),
                                       setattr(d, "global_stride", 1)), "ATTN_ERR_BAD_VARIANT"),
    ("heads per wg 3", lambda d: setattr(d, "sched_heads_per_wg", 3), "ATTN_ERR_BAD_VARIANT"),
    ("heads per wg 8", lambda d: setattr(d, "sched_heads_per_wg", 8), "ATTN_ERR_BAD_VARIANT"),
    ("heads per wg not dividing", lambda d: (setattr(d, "num_q_heads", 6), setattr(d, "num_kv_heads", 3),
                                             setattr(d, "sched_heads_per_wg", 4)),
     "ATTN_ERR_BAD_VARIANT"),
    ("heads per wg fp32", lambda d: (setattr(d, "dtype", _abi.ATTN_FP32), setattr(d, "sched_heads_per_wg", 2)),
     "ATTN_ERR_BAD_VARIANT"),
    ("order 3", lambda d: setattr(d, "sched_order", 3), "ATTN_ERR_BAD_VARIANT"),
    ("xcd order needs B*Hkv % 8", lambda d: setattr(d, "sched_order", 2), "ATTN_ERR_BAD_VARIANT"),
    ("chunk with natural order", lambda d: (setattr(d, "sched_order", 1), setattr(d, "sched_chunk", 1)),
     "ATTN_ERR_BAD_VARIANT"),
    ("chunk without xcd order", lambda d: setattr(d, "sched_chunk", 1), "ATTN_ERR_BAD_VARIANT"),
    ("chunk beyond groups", lambda d: (setattr(d, "batch", 4), setattr(d, "sched_chunk", 2)),
     "ATTN_ERR_BAD_VARIANT"),
    ("negative chunk", lambda d: setattr(d, "sched_chunk", -1), "ATTN_ERR_BAD_VARIANT"),
    # output rows must be disjoint: heads on top of each other, or rows that
    # overlap the next head
    ("out heads overlap", lambda d: setattr(d, "stride_o_h", 128), "ATTN_ERR_BAD_SHAPE"),
    ("out head stride below D", lambda d: setattr(d, "stride_o_h", 64), "ATTN_ERR_BAD_SHAPE"),
    ("out rows run into the next head", lambda d: setattr(d, "stride_o_h", 99 * 128),
     "ATTN_ERR_BAD_SHAPE"),
    ("out batches overlap", lambda d: setattr(d, "stride_o_b", 8 * 100 * 128 - 8),
     "ATTN_ERR_BAD_SHAPE"),
]


@pytest.mark.parametrize("name,mutate,expect", CASES, ids=[c[0] for c in CASES])
def test_validation_errors(lib, name, mutate, expect):
    d = base_desc()
    mutate(d)
    assert call(lib, d) == err(expect)


VARLEN_CASES = [
    ("cu_k missing", lambda d: setattr(d, "cu_seqlens_k", None), "ATTN_ERR_NULL_PTR"),
    ("out token stride below the heads", lambda d: setattr(d, "stride_o_s", 4 * 128),
     "ATTN_ERR_BAD_SHAPE"),
    ("out head stride below D", lambda d: setattr(d, "stride_o_h", 64), "ATTN_ERR_BAD_SHAPE"),
    ("max_seqlen < 0", lambda d: setattr(d, "max_seqlen_q", -1), "ATTN_ERR_BAD_SHAPE"),
    ("total < 0", lambda d: setattr(d, "total_k", -1), "ATTN_ERR_BAD_SHAPE"),
    ("total beyond int32", lambda d: setattr(d, "total_q", 1 << 33), "ATTN_ERR_UNSUPPORTED"),
]


@pytest.mark.parametrize("name,mutate,expect", VARLEN_CASES, ids=[c[0] for c in VARLEN_CASES])
def test_varlen_validation_errors(lib, name, mutate, expect):
    d = base_desc(varlen=True)
    mutate(d)
    assert call(lib, d) == err(expect)


def test_pointer_errors(lib):
    assert call(lib, None) == err("ATTN_ERR_NULL_PTR")
    d = base_desc()
    for kw in ({"q": None}, {"k": None}, {"v": None}, {"o": None}):
        assert call(lib, d, **kw) == err("ATTN_ERR_NULL_PTR")
    for kw in ({"q": P + 2}, {"k": P + 8}, {"v": P + 4}, {"o": P + 1}):
        assert call(lib, d, **kw) == err("ATTN_ERR_ALIGNMENT")
    assert call(lib, d, lse=P + 2) == err("ATTN_ERR_ALIGNMENT")


def test_fp32_alignment_unit(lib):
    d = base_desc()
    d.dtype = _abi.ATTN_FP32
    d.stride_q_s = 132  # 4-element multiple: fine for fp32 ...
    d.stride_q_h = 132 * 100
    d.stride_q_b = 132 * 100 * 8
    d.seqlen_q = 0       # ... and an empty problem returns before any launch
    assert call(lib, d) == 0
    d.stride_q_s = 130   # not a multiple of 4 fp32 elements
    assert call(lib, d) == err("ATTN_ERR_ALIGNMENT")


def test_empty_problems_do_nothing(lib):
    for mut in (lambda d: setattr(d, "batch", 0), lambda d: setattr(d, "seqlen_q", 0)):
        d = base_desc()
        mut(d)
        assert call(lib, d, q=None, k=None, v=None, o=None, lse=None) == 0
    d = base_desc(varlen=True)
    d.max_seqlen_q = 0
    assert call(lib, d, q=None, k=None, v=None, o=None, lse=None) == 0


def test_disjoint_strided_outputs_accepted(lib):
    """Interleaved but disjoint output layouts pass the overlap check."""
    for mut in (lambda d: (setattr(d, "stride_o_s", 8 * 128), setattr(d, "stride_o_h", 128),
                           setattr(d, "stride_o_b", 100 * 8 * 128)),   # [B, S, H, D]
                lambda d: (setattr(d, "stride_o_s", 136), setattr(d, "stride_o_h", 100 * 136),
                           setattr(d, "stride_o_b", 8 * 100 * 136))):  # padded rows
        d = base_desc()
        mut(d)
        # the overlap check passes, so the call reaches the pointer check (a
        # rejected layout would return ATTN_ERR_BAD_SHAPE before it)
        assert call(lib, d, q=None) == err("ATTN_ERR_NULL_PTR")


def test_broadcast_inputs_accepted(lib):
    """Inputs may overlap (a K/V head broadcast with stride 0 is read only)."""
    d = base_desc()
    d.stride_k_h = 0
    d.stride_v_h = 0
    assert call(lib, d, q=None) == err("ATTN_ERR_NULL_PTR")


def test_row_range_rejects_listed_global_set(lib):
    d = base_desc()
    d.mask_kind = _abi.ATTN_MASK_GLOBAL_SLIDING_WINDOW
    d.window_left = d.window_right = 4
    d.num_global = 3
    d.global_tokens = P  # never dereferenced
    out = (ctypes.c_int32 * 3)()
    assert lib.attn_row_range(ctypes.byref(d), None, 0, 10, 10, out) == err("ATTN_ERR_UNSUPPORTED")
    d.global_tokens = None  # leading run: prefix plus band
    assert lib.attn_row_range(ctypes.byref(d), None, 5, 10, 10, out) == 0
    assert tuple(out) == (0, 0, 9)  # prefix {0,1,2} touches the band [1, 9]: merged


def test_per_sequence_layout_strides_accepted(lib):
    """A stride of at least the entry count (one row per sequence) passes the
    host checks and the call reaches the pointer check."""
    d = base_desc()
    d.mask_kind = _abi.ATTN_MASK_SHARE_QUESTION
    d.segment_starts = P
    d.num_segments = 3
    d.segment_stride = 3
    assert call(lib, d, q=None) == err("ATTN_ERR_NULL_PTR")
    d.segment_stride = 16  # padded rows
    assert call(lib, d, q=None) == err("ATTN_ERR_NULL_PTR")
    d = base_desc()
    d.mask_kind = _abi.ATTN_MASK_GLOBAL_SLIDING_WINDOW
    d.window_left = d.window_right = 4
    d.global_tokens = P
    d.num_global = 5
    d.global_stride = 5
    assert call(lib, d, q=None) == err("ATTN_ERR_NULL_PTR")

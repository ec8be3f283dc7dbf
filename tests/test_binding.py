"""The Python binding on the CPU: every shape, dtype and device mismatch
between q and the other tensors raises before anything reaches the C ABI
(which sees only pointers, so a mismatch there would read or write past the
caller's buffers). CPU tensors stand in for device tensors: make_desc builds
the descriptor without launching anything."""
import pytest
import torch

import paper_2605_05023_amd as attn


def T(*shape, dtype=torch.bfloat16):
    return torch.zeros(shape, dtype=dtype)


def fixed(**over):
    t = dict(q=T(2, 8, 100, 128), k=T(2, 2, 120, 128), v=T(2, 2, 120, 128),
             out=T(2, 8, 100, 128))
    t.update(over)
    return t


def packed(**over):
    t = dict(q=T(150, 8, 64), k=T(170, 2, 64), v=T(170, 2, 64), out=T(150, 8, 64))
    t.update(over)
    return t


CU = torch.tensor([0, 100, 150], dtype=torch.int32)
CUK = torch.tensor([0, 120, 170], dtype=torch.int32)


def desc(t, **kw):
    return attn.make_desc(t["q"], t["k"], t["v"], t["out"], stream=0, **kw)


def varlen_desc(t, **kw):
    base = dict(cu_seqlens_q=CU, cu_seqlens_k=CUK, max_seqlen_q=100, max_seqlen_k=120)
    base.update(kw)
    return desc(t, **base)


def test_well_formed_inputs_build_a_descriptor():
    d = desc(fixed(), causal=True)
    assert (d.batch, d.num_q_heads, d.num_kv_heads, d.seqlen_q, d.seqlen_k) == (2, 8, 2, 100, 120)
    d = varlen_desc(packed(), alibi_slopes=torch.ones(8))
    assert (d.batch, d.total_q, d.total_k, d.head_dim) == (2, 150, 170, 64)
    d = desc(fixed(), validate=True, heads_per_wg=2, order="xcd_groups", chunk=1)
    assert (d.flags, d.sched_heads_per_wg, d.sched_order, d.sched_chunk) == (1, 2, 2, 1)


FIXED_BAD = [
    ("k head dim", dict(k=T(2, 2, 120, 64), v=T(2, 2, 120, 64))),
    ("v head dim", dict(v=T(2, 2, 120, 64))),
    ("k and v lengths", dict(v=T(2, 2, 119, 128))),
    ("k and v heads", dict(v=T(2, 4, 120, 128))),
    ("k batch", dict(k=T(1, 2, 120, 128), v=T(1, 2, 120, 128))),
    ("out shape", dict(out=T(2, 8, 99, 128))),
    ("out heads", dict(out=T(2, 4, 100, 128))),
    ("q rank", dict(q=T(8, 100, 128), out=T(8, 100, 128))),
    ("k rank", dict(k=T(2, 120, 128), v=T(2, 120, 128))),
]


@pytest.mark.parametrize("name,over", FIXED_BAD, ids=[c[0] for c in FIXED_BAD])
def test_fixed_length_shape_mismatch_raises(name, over):
    with pytest.raises(ValueError):
        desc(fixed(**over))


def test_slopes_checked():
    with pytest.raises(ValueError):
        desc(fixed(), alibi_slopes=torch.ones(7))
    with pytest.raises(TypeError):
        desc(fixed(), alibi_slopes=torch.ones(8, dtype=torch.float64))
    with pytest.raises(TypeError):
        desc(fixed(), alibi_slopes=torch.ones(16)[::2])


def test_dtype_mismatch_raises():
    with pytest.raises(TypeError):
        desc(fixed(k=T(2, 2, 120, 128, dtype=torch.float32)))
    with pytest.raises(TypeError):
        desc(fixed(out=T(2, 8, 100, 128, dtype=torch.float16)))


def test_innermost_axis_must_be_contiguous():
    q = T(2, 8, 128, 100).transpose(-1, -2)
    with pytest.raises(ValueError):
        desc(fixed(q=q))


PACKED_BAD = [
    ("k head dim", dict(k=T(170, 2, 128), v=T(170, 2, 128))),
    ("k and v tokens", dict(v=T(160, 2, 64))),
    ("out tokens", dict(out=T(149, 8, 64))),
    ("out heads", dict(out=T(150, 4, 64))),
    ("q rank", dict(q=T(1, 150, 8, 64), out=T(1, 150, 8, 64))),
]


@pytest.mark.parametrize("name,over", PACKED_BAD, ids=[c[0] for c in PACKED_BAD])
def test_packed_shape_mismatch_raises(name, over):
    with pytest.raises(ValueError):
        varlen_desc(packed(**over))


def test_cu_seqlens_checked():
    with pytest.raises(ValueError):  # different numbers of sequences
        varlen_desc(packed(), cu_seqlens_k=torch.tensor([0, 170], dtype=torch.int32))
    with pytest.raises(TypeError):
        varlen_desc(packed(), cu_seqlens_q=CU.long())
    with pytest.raises(ValueError):
        varlen_desc(packed(), max_seqlen_k=None)


def test_index_arrays_checked():
    with pytest.raises(TypeError):
        desc(fixed(), mask="share_question", segment_starts=torch.tensor([3, 9]))
    with pytest.raises(ValueError):
        desc(fixed(), mask="global_sliding_window", window=(4, 4), num_global=3,
             global_tokens=torch.tensor([0, 5], dtype=torch.int32))
    d = desc(fixed(), mask="global_sliding_window", window=(4, 4),
             global_tokens=torch.tensor([0, 5, 90], dtype=torch.int32))
    assert d.num_global == 3 and d.global_tokens


def test_lse_shape():
    assert attn.lse_shape(T(2, 8, 100, 128), False) == (2, 8, 100)
    assert attn.lse_shape(T(150, 8, 64), True) == (8, 150)


def test_fwd_refuses_host_tensors():
    t = fixed()
    with pytest.raises(ValueError):
        attn.fwd(t["q"], t["k"], t["v"], causal=True)


def test_per_sequence_layouts():
    """segment_starts / global_tokens: one array shared by every sequence, or
    one row per sequence ([batch, n]) whose row stride becomes the
    descriptor's stride."""
    seg = torch.tensor([10, 20, 30], dtype=torch.int32)
    d = desc(fixed(), mask="share_question", segment_starts=seg)
    assert (d.num_segments, d.segment_stride) == (3, 0)
    rows = torch.tensor([[10, 20, 30], [5, 6, 99]], dtype=torch.int32)
    d = desc(fixed(), mask="causal_blockwise", segment_starts=rows)
    assert (d.num_segments, d.segment_stride) == (3, 3)
    padded = torch.zeros((2, 8), dtype=torch.int32)[:, :3]  # rows 8 apart
    d = desc(fixed(), mask="share_question", segment_starts=padded)
    assert (d.num_segments, d.segment_stride) == (3, 8)
    g = torch.tensor([[0, 50], [3, 7]], dtype=torch.int32)
    d = varlen_desc(packed(), mask="global_sliding_window", window=(4, 4), global_tokens=g)
    assert (d.num_global, d.global_stride) == (2, 2)


PERSEQ_BAD = [
    ("rows != batch", dict(mask="share_question",
                           segment_starts=torch.zeros((3, 2), dtype=torch.int32)), ValueError),
    ("rank 3", dict(mask="share_question",
                    segment_starts=torch.zeros((2, 2, 2), dtype=torch.int32)), ValueError),
    ("column-major rows", dict(mask="share_question",
                               segment_starts=torch.zeros((4, 2), dtype=torch.int32).t()),
     ValueError),
    ("global rows != batch", dict(mask="global_sliding_window", window=(4, 4),
                                  global_tokens=torch.zeros((1, 2), dtype=torch.int32)), ValueError),
    ("int64 rows", dict(mask="share_question", segment_starts=torch.zeros((2, 2))), TypeError),
]


@pytest.mark.parametrize("name,kw,exc", PERSEQ_BAD, ids=[c[0] for c in PERSEQ_BAD])
def test_per_sequence_layout_errors(name, kw, exc):
    with pytest.raises(exc):
        desc(fixed(), **kw)


def test_log_flag():
    d = desc(fixed(), causal=True, log=True)
    assert d.flags == attn.ATTN_FLAG_LOG
    d = desc(fixed(), causal=True, log=True, validate=True)
    assert d.flags == attn.ATTN_FLAG_LOG | attn.ATTN_FLAG_VALIDATE

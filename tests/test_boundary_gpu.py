"""GPU behaviour at the C-ABI boundary: strided views in and out, a NULL LSE,
a non-default stream, bitwise determinism across calls, and no writes outside
the output rows (guard regions around O and LSE)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_05023_amd as attn
from gpu_util import assert_parity, gpu_available, log
from paper_2605_05023_amd.workloads import MASK_CAUSAL, MASK_SLIDING_WINDOW, Workload, make_inputs

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = torch.device("cuda:0")


def _bshd_views(t):
    """A [B, S, H, D] contiguous copy of a [B, H, S, D] tensor, returned as a
    [B, H, S, D] view (strides b = S*H*D, h = D, s = H*D)."""
    return t.permute(0, 2, 1, 3).contiguous().to(DEV).permute(0, 2, 1, 3)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_strided_views_in_and_out(dtype):
    wl = Workload("strided", dtype, 2, 4, 2, 200, 64, mask=MASK_CAUSAL, seed=31)
    inp = make_inputs(wl)
    q, k, v = _bshd_views(inp.q), _bshd_views(inp.k), _bshd_views(inp.v)
    assert not q.is_contiguous() and q.stride(1) == 64
    # output into a padded buffer: [B, S, H, D + 8] sliced to D, viewed as BHSD
    buf = torch.full((2, 200, 4, 72), math.nan, dtype=q.dtype, device=DEV)
    out = buf[..., :64].permute(0, 2, 1, 3)
    o, lse = attn.fwd(q, k, v, causal=True, out=out, scale=wl.scale)
    torch.cuda.synchronize()
    assert o.data_ptr() == out.data_ptr()
    assert torch.isnan(buf[..., 64:].float()).all(), "wrote into the padding"
    log(f"[boundary] strided {dtype}")
    assert_parity(inp, o, lse, label=f"strided {dtype}")


def test_varlen_token_stride():
    # tokens padded to 2*D elements: head stride 2D... token stride H*2D
    wl = Workload("varlen_stride", "bf16", 3, 4, 2, 0, 64, mask=MASK_CAUSAL, seed=32,
                  varlen=True)
    inp = make_inputs(wl, lengths=[100, 0, 170])

    def padded(t):
        T, H, D = t.shape
        big = torch.zeros((T, H, 2 * D), dtype=t.dtype)
        big[..., :D] = t
        return big.to(DEV)[..., :D]
    q, k, v = padded(inp.q), padded(inp.k), padded(inp.v)
    assert q.stride() == (4 * 128, 128, 1)
    cu = inp.cu_seqlens.to(DEV)
    o, lse = attn.fwd(q, k, v, causal=True, cu_seqlens_q=cu, cu_seqlens_k=cu,
                      max_seqlen_q=inp.max_seqlen, max_seqlen_k=inp.max_seqlen, scale=wl.scale)
    assert_parity(inp, o, lse, label="varlen token stride")


def test_null_lse_and_stream():
    wl = Workload("stream", "bf16", 1, 4, 4, 300, 128, mask=MASK_SLIDING_WINDOW,
                  window_left=40, window_right=0, seed=33)
    inp = make_inputs(wl)
    s = torch.cuda.Stream()  # default priority
    with torch.cuda.stream(s):
        q, k, v = inp.q.to(DEV), inp.k.to(DEV), inp.v.to(DEV)
        o1 = attn.fwd(q, k, v, window=(40, 0), scale=wl.scale, return_lse=False)
        o2, lse = attn.fwd(q, k, v, window=(40, 0), scale=wl.scale)
    s.synchronize()
    assert torch.equal(o1, o2), "O differs with and without LSE"
    assert_parity(inp, o2, lse, label="side stream")


def test_deterministic_and_guarded():
    """Two calls give bitwise-equal O and LSE; nothing outside O and LSE changes."""
    wl = Workload("guard", "bf16", 2, 4, 4, 257, 128, mask=MASK_CAUSAL, seed=34)
    inp = make_inputs(wl)
    q, k, v = inp.q.to(DEV), inp.k.to(DEV), inp.v.to(DEV)
    n_o, n_l = q.numel(), 2 * 4 * 257
    obuf = torch.full((n_o + 4096,), math.nan, dtype=torch.bfloat16, device=DEV)
    lbuf = torch.full((n_l + 1024,), math.nan, dtype=torch.float32, device=DEV)
    out = obuf[2048:2048 + n_o].view(q.shape)
    lse = lbuf[512:512 + n_l].view(2, 4, 257)
    attn.fwd(q, k, v, causal=True, out=out, lse=lse, scale=wl.scale)
    o1, l1 = out.clone(), lse.clone()
    attn.fwd(q, k, v, causal=True, out=out, lse=lse, scale=wl.scale)
    torch.cuda.synchronize()
    assert torch.equal(out, o1) and torch.equal(lse, l1), "not bitwise deterministic"
    for b, lo, hi in ((obuf, 2048, 2048 + n_o), (lbuf, 512, 512 + n_l)):
        assert torch.isnan(b[:lo].float()).all() and torch.isnan(b[hi:].float()).all(), \
            "write outside the output"
    assert_parity(inp, out, lse, label="guarded")


def test_lse_combines_key_shards():
    """Attention over keys [0, Sk) equals the LSE-weighted merge of attention over
    two key shards (the split a sequence-sharded run would merge), both shards
    computed by the kernel with bottom-right-free (non-causal) masks."""
    wl = Workload("shards", "bf16", 1, 2, 2, 256, 128, seed=35)
    inp = make_inputs(wl)
    q, k, v = inp.q.to(DEV), inp.k.to(DEV), inp.v.to(DEV)
    o, lse = attn.fwd(q, k, v, scale=wl.scale)
    parts = [attn.fwd(q, k[:, :, a:b].contiguous(), v[:, :, a:b].contiguous(), scale=wl.scale)
             for a, b in ((0, 100), (100, 256))]
    lses = torch.stack([p[1] for p in parts])
    m = torch.logsumexp(lses, 0)
    merged = sum(torch.exp(p[1] - m)[..., None] * p[0].float() for p in parts)
    err_o = (merged - o.float()).abs().max().item()
    err_l = (m - lse).abs().max().item()
    log(f"[boundary] shard merge: max|dO| {err_o:.3e}, max|dLSE| {err_l:.3e}")
    assert err_o <= 2e-2 and err_l <= 1e-3

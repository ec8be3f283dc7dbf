"""GPU behaviour at the C-ABI boundary: strided views in and out, a NULL LSE,
a non-default stream, bitwise determinism across calls, no writes outside
the output rows (guard regions around O and LSE), and the largest slices and
offsets the 32-bit in-slice addressing allows."""
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


def test_concurrent_streams():
    """Calls on two streams interleaved without a host wait between them (a
    causal bf16 problem and a packed ALiBi + soft-cap one, launched in turn
    four times each) give bit for bit the outputs of the same calls run alone:
    the library keeps no state between calls."""
    wa = Workload("conc_a", "bf16", 2, 8, 2, 700, 128, mask=MASK_CAUSAL, seed=36)
    wb = Workload("conc_b", "bf16", 3, 4, 4, 0, 64, mask=MASK_CAUSAL, alibi=True, softcap=30.0,
                  seed=37, varlen=True)
    ia, ib = make_inputs(wa), make_inputs(wb, lengths=[500, 17, 900])
    ka, kb = ia.variant_kwargs(DEV), ib.variant_kwargs(DEV)
    qa, kva = ia.q.to(DEV), (ia.k.to(DEV), ia.v.to(DEV))
    qb, kvb = ib.q.to(DEV), (ib.k.to(DEV), ib.v.to(DEV))
    ref_a = attn.fwd(qa, *kva, **ka)
    ref_b = attn.fwd(qb, *kvb, **kb)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()  # default priority
    outs = []
    for _ in range(4):
        with torch.cuda.stream(sa):
            oa = attn.fwd(qa, *kva, **ka)
        with torch.cuda.stream(sb):
            ob = attn.fwd(qb, *kvb, **kb)
        outs.append((oa, ob))
    sa.synchronize()
    sb.synchronize()
    log("[boundary] two streams interleaved, 4 rounds")
    for (oa, la), (ob, lb) in outs:
        assert torch.equal(oa, ref_a[0]) and torch.equal(la, ref_a[1])
        assert torch.equal(ob, ref_b[0]) and torch.equal(lb, ref_b[1])
    assert_parity(ia, ref_a[0], ref_a[1], label="concurrent a")
    assert_parity(ib, ref_b[0], ref_b[1], label="concurrent b")


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


def _tail_case(sq, tail, seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((sq, 128), generator=g).to(torch.bfloat16)
    kt = torch.randn((tail, 128), generator=g).to(torch.bfloat16)
    vt = torch.randn((tail, 128), generator=g).to(torch.bfloat16)
    return q, kt, vt


def _check(o, lse, o_ref, lse_ref, label):
    err_o = float(np.abs(o.float().cpu().numpy() - o_ref).max())
    err_l = float(np.abs(lse.cpu().numpy().astype(np.float64) - lse_ref).max())
    log(f"[boundary] {label}: max|dO| {err_o:.3e}, max|dLSE| {err_l:.3e}")
    assert err_o <= 2e-2 and err_l <= 1e-3


def test_largest_slice():
    """One head whose K/V slice is the largest the host accepts (its last byte
    just below 2^31 with one tile of padding): 128 queries bottom-right aligned
    against 8,388,478 keys under a 200-key causal window, so only keys at the
    very end of the slice are visible. Every other key is zero; the oracle
    runs on the last 4096 keys, which bottom-right alignment makes the same
    problem."""
    sk, sq, tail, wl = (1 << 23) - 130, 128, 4096, 200
    q, kt, vt = _tail_case(sq, tail, 41)
    k = torch.zeros((1, 1, sk, 128), dtype=torch.bfloat16, device=DEV)
    v = torch.zeros((1, 1, sk, 128), dtype=torch.bfloat16, device=DEV)
    k[0, 0, sk - tail:] = kt.to(DEV)
    v[0, 0, sk - tail:] = vt.to(DEV)
    log(f"[boundary] largest slice: Sk={sk} ({2 * sk * 128 * 2 / 2**30:.2f} GiB of K/V)")
    o, lse = attn.fwd(q.view(1, 1, sq, 128).to(DEV), k, v, window=(wl, 0), scale=128 ** -0.5)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.attention(q.view(1, 1, sq, 128), kt.view(1, 1, tail, 128),
                                      vt.view(1, 1, tail, 128), scale=128 ** -0.5,
                                      mask=MASK_SLIDING_WINDOW, window_left=wl, window_right=0)
    _check(o, lse, o_ref, lse_ref, "largest slice")
    del k, v
    torch.cuda.empty_cache()


def test_sequence_beyond_2gib():
    """Packed batch whose third sequence starts 2.3 GB into K and V (the
    first two have 4,500,000 keys each and no queries): the slice base is
    formed with 64-bit arithmetic, offsets inside a slice stay 32-bit."""
    n0, sq, tail = 9_000_000, 200, 300
    q, kt, vt = _tail_case(sq, tail, 42)
    tk = n0 + tail
    k = torch.zeros((tk, 1, 128), dtype=torch.bfloat16, device=DEV)
    v = torch.zeros((tk, 1, 128), dtype=torch.bfloat16, device=DEV)
    k[n0:, 0] = kt.to(DEV)
    v[n0:, 0] = vt.to(DEV)
    cuq = torch.tensor([0, 0, 0, sq], dtype=torch.int32)
    cuk = torch.tensor([0, n0 // 2, n0, tk], dtype=torch.int32)
    log(f"[boundary] sequence at {n0 * 256 / 1e9:.2f} GB into K/V")
    o, lse = attn.fwd(q.view(sq, 1, 128).to(DEV), k, v, causal=True, cu_seqlens_q=cuq.to(DEV),
                      cu_seqlens_k=cuk.to(DEV), max_seqlen_q=sq, max_seqlen_k=n0 // 2,
                      scale=128 ** -0.5)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.attention(q.view(1, 1, sq, 128), kt.view(1, 1, tail, 128),
                                      vt.view(1, 1, tail, 128), scale=128 ** -0.5,
                                      mask=MASK_CAUSAL)
    _check(o.view(1, sq, 1, 128).permute(0, 2, 1, 3), lse.view(1, 1, sq), o_ref, lse_ref,
           "sequence beyond 2 GiB")
    del k, v
    torch.cuda.empty_cache()

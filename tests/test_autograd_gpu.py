"""torch autograd through the kernels: swin_attention's gradients equal those of the explicit
training forward + backward calls (same kernels, same inputs: bitwise), for bf16 and fp32,
both padding modes, a multi-scale grid list and fused RoPE; and a non-contiguous input gets
its gradient in its own layout."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2407_02109_amd import binding as fb
from paper_2407_02109_amd import synth

pytestmark = pytest.mark.gpu


def _say(msg):
    print("[case] %s" % msg, flush=True)


def _leaf(t):
    return t.cuda().detach().requires_grad_(True)


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_autograd_matches_explicit_calls(dtype, pm):
    _say("autograd %s pm=%d" % (dtype, pm))
    wl = synth.Workload("ag", 2, 3, 37, 29, 64, 16, 8, dtype, seed=77 + pm, pad_mode=pm)
    q, k, v = (_leaf(t) for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    out = fb.swin_attention(q, k, v, [(wl.H, wl.W)], wl.window, wl.shift, pm)
    out.backward(dout)
    with torch.no_grad():
        o2, lse = fb.swin_attn_fwd_train(q.detach(), k.detach(), v.detach(), [(wl.H, wl.W)], wl.window, wl.shift, pm)
        g2 = fb.swin_attn_bwd(q.detach(), k.detach(), v.detach(), o2, dout, lse, [(wl.H, wl.W)], wl.window,
                              wl.shift, pm)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), o2)
    for got, ref in zip((q.grad, k.grad, v.grad), g2):
        assert torch.equal(got, ref)


def test_autograd_multiscale_and_oracle():
    _say("autograd multi-scale")
    grids = [(40, 24), (8, 8)]
    L = sum(h * w for h, w in grids)
    g = torch.Generator().manual_seed(5)
    q, k, v, dout = (torch.randn(1, L + (1 if i in (1, 2) else 0), 2, 64, generator=g).to(torch.bfloat16)
                     for i in range(4))
    qd, kd, vd = _leaf(q), _leaf(k), _leaf(v)
    out = fb.swin_attention(qd, kd, vd, grids, 16, 8, 1)
    out.backward(dout.cuda())
    torch.cuda.synchronize()
    refs = O.swin_attention_ms_bwd(*(synth.to_f64_numpy(t) for t in (q, k, v, dout)), grids, 16, 8, 1)
    for got, ref in zip((qd.grad, kd.grad, vd.grad), refs):
        got = synth.to_f64_numpy(got)
        m = np.abs(ref).max()
        assert np.abs(got - ref).max() <= 2e-2 * m and np.abs(got - ref).mean() <= 2e-3 * m


def test_autograd_rope_matches_explicit_calls():
    _say("autograd rope")
    wl = synth.Workload("agr", 1, 2, 20, 13, 64, 8, 3, "bf16", seed=9, pad_mode=1)
    q, k, v = (_leaf(t) for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    rope = (100.0, 0.5)
    out = fb.swin_attention(q, k, v, [(wl.H, wl.W)], wl.window, wl.shift, 1, rope=rope)
    out.backward(dout)
    with torch.no_grad():
        o2, lse = fb.swin_attn_rope_fwd_train(q.detach(), k.detach(), v.detach(), wl.H, wl.W, wl.window, wl.shift,
                                              1, *rope)
        g2 = fb.swin_attn_rope_bwd(q.detach(), k.detach(), v.detach(), o2, dout, lse, wl.H, wl.W, wl.window,
                                   wl.shift, 1, *rope)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), o2)
    for got, ref in zip((q.grad, k.grad, v.grad), g2):
        assert torch.equal(got, ref)


def test_autograd_non_contiguous_input():
    _say("autograd non-contiguous")
    wl = synth.Workload("agn", 1, 2, 16, 16, 64, 8, 4, "bf16", seed=13)
    q, k, v = synth.make_inputs(wl)
    # q as a transposed view of a [B, heads, L, 64] leaf
    base = q.permute(0, 2, 1, 3).contiguous().cuda().requires_grad_(True)
    qv = base.permute(0, 2, 1, 3)
    assert not qv.is_contiguous()
    kd, vd = _leaf(k), _leaf(v)
    dout = synth.make_grad(wl).cuda()
    out = fb.swin_attention(qv, kd, vd, [(16, 16)], 8, 4, 0)
    out.backward(dout)
    qc = _leaf(q)
    out2 = fb.swin_attention(qc, _leaf(k), _leaf(v), [(16, 16)], 8, 4, 0)
    out2.backward(dout)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), out2.detach())
    assert torch.equal(base.grad.permute(0, 2, 1, 3), qc.grad)

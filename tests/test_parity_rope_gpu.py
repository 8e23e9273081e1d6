"""GPU parity of the forward with 2-D RoPE fused into its prologue, against the fp64 oracle
(``oracle.rope``: q and k rotated in fp64, then the textbook attention).

Tolerances as for the plain forward: bf16 max-abs 2e-2 and mean-abs 2e-3, fp32 max-abs
1e-5.  The bf16 kernel rotates the loaded bf16 values in fp32 and rounds them back to bf16
before the products (one more rounding of q and k, relative 2^-9), with the hardware sine
on the angle reduced to half a revolution; the fp32 kernel computes the angles and their
sine and cosine in double."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2407_02109_amd import binding as fb
from paper_2407_02109_amd import synth

pytestmark = pytest.mark.gpu

BF16_MAX, BF16_MEAN, F32_MAX = 2e-2, 2e-3, 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fb.load_library()


def _say(msg):
    print("[case] %s" % msg, flush=True)


def _compare(got, ref, f32):
    got = synth.to_f64_numpy(got)
    assert np.isfinite(got).all(), "non-finite output (unwritten rows?)"
    err = np.abs(got - ref)
    if f32:
        assert err.max() <= F32_MAX, err.max()
    else:
        assert err.max() <= BF16_MAX and err.mean() <= BF16_MEAN, (err.max(), err.mean())


SHAPES = [  # B, heads, H, W, window, shift
    (2, 2, 64, 64, 16, 8), (1, 3, 37, 29, 16, 8), (2, 2, 20, 13, 8, 3), (1, 1, 9, 7, 16, 0),
    (1, 1, 9, 300, 16, 15), (1, 1, 1, 1, 1, 0), (1, 2, 40, 24, 32, 16),
]
ROPES = [(10000.0, 1.0), (100.0, 0.5)]


@pytest.mark.parametrize("rope", ROPES, ids=["theta1e4", "theta100_half"])
@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_rope_forward(shape, dtype, pm, rope):
    B, heads, H, W, k, s = shape
    _say("rope %s %s pad_mode=%d rope=%s" % (shape, dtype, pm, rope))
    wl = synth.Workload("case", B, heads, H, W, 64, k, s, dtype, seed=200 + sum(shape) + pm, pad_mode=pm)
    q, kk, v = synth.make_inputs(wl)
    out = torch.full_like(q, float("nan"), device="cuda")
    fb.fla_swin_attn_rope_fwd(q.cuda(), kk.cuda(), v.cuda(), out, B, heads, H, W, 64, k, s, pm, rope[0], rope[1],
                              f32=dtype == "f32")
    torch.cuda.synchronize()
    ref = O.swin_attention_rope(*(synth.to_f64_numpy(t) for t in (q, kk, v)), H, W, k, s, pm, rope[0], rope[1])
    _compare(out, ref, dtype == "f32")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rope_scale_zero_is_the_plain_forward(dtype):
    wl = synth.Workload("case", 1, 2, 37, 29, 64, 16, 8, dtype, seed=9, pad_mode=1)
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    a, b = torch.empty_like(q), torch.empty_like(q)
    f32 = dtype == "f32"
    fb.fla_swin_attn_rope_fwd(q, kk, v, a, 1, 2, 37, 29, 64, 16, 8, 1, 10000.0, 0.0, f32=f32)
    (fb.fla_swin_attn_fwd_f32 if f32 else fb.fla_swin_attn_fwd)(q, kk, v, b, 1, 2, 37, 29, 64, 16, 8, 1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_full_size_rope_sampled():
    wl = synth.WORKLOADS["img4096_rope"]
    _say("rope full size img4096_rope")
    q, kk, v = synth.make_inputs(wl)
    out = torch.full_like(q, float("nan"), device="cuda")
    theta, scale = wl.rope
    qd, kd, vd = q.cuda(), kk.cuda(), v.cuda()
    fb.fla_swin_attn_rope_fwd(qd, kd, vd, out, wl.B, wl.heads, wl.H, wl.W, 64, wl.window, wl.shift, wl.pad_mode,
                              theta, scale)
    out2 = torch.empty_like(out)
    fb.fla_swin_attn_rope_fwd(qd, kd, vd, out2, wl.B, wl.heads, wl.H, wl.W, 64, wl.window, wl.shift, wl.pad_mode,
                              theta, scale)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    got = synth.to_f64_numpy(out)
    assert np.isfinite(got).all()
    pts = synth.random_queries(wl, 300, seed=17).numpy()
    ref = O.swin_attention_rope_at(*(synth.to_f64_numpy(t) for t in (q, kk, v)), wl.H, wl.W, wl.window, wl.shift,
                                   wl.pad_mode, pts, theta, scale)
    sel = got[pts[:, 0], pts[:, 1] * wl.W + pts[:, 2]]
    err = np.abs(sel - ref)
    assert err.max() <= BF16_MAX and err.mean() <= BF16_MEAN, (err.max(), err.mean())

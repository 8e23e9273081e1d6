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
    # windows wider than the bf16 kernel's 32 x 32 cos / sin table: (cos, sin) per rotated
    # piece; the second mixes 20 x 20 windows (table) with 40 x 40 ones (direct)
    (1, 1, 40, 24, 40, 0), (1, 2, 64, 64, 40, 20),
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


# ---- RoPE training: forward with log-sum-exp, backward (gradients of the unrotated q, k, v)
BWD_SHAPES = [(2, 2, 64, 64, 16, 8), (1, 3, 37, 29, 16, 8), (2, 2, 20, 13, 8, 3), (1, 1, 9, 300, 16, 15),
              # windows over 256 tokens; the last three also wider than 32 rows or columns
              (1, 2, 40, 37, 20, 10), (1, 1, 40, 40, 32, 16), (1, 1, 40, 24, 40, 0), (1, 2, 64, 64, 40, 20),
              (1, 1, 64, 64, 64, 0)]


def _check_grad(name, got, ref, f32, bulk=True):
    """Gradient bounds relative to M = max |reference| (as for the plain backward)."""
    got = synth.to_f64_numpy(got)
    assert np.isfinite(got).all(), name
    M = np.abs(ref).max()
    err = np.abs(got - ref)
    if f32:
        assert err.max() <= F32_MAX * M, (name, err.max() / M)
    else:
        assert err.max() <= BF16_MAX * M, (name, err.max() / M)
        if bulk:
            assert err.mean() <= BF16_MEAN * M, (name, err.mean() / M)


# fp32 RoPE training is withdrawn: its first GPU run (the fp32 backward kernels with the
# rotation added, which made them use 528 bytes of scratch per lane) ended in a GPU memory
# fault, while the same sources run on the CPU stayed in bounds and matched the oracle.
# Without a cause shown the fp32 path is not offered and these cases stay skipped.
_F32_WITHDRAWN = pytest.mark.skip(reason="fp32 RoPE training withdrawn: its first GPU run faulted, cause not "
                                         "found (sources in bounds on the CPU)")


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
@pytest.mark.parametrize("dtype", ["bf16", pytest.param("f32", marks=_F32_WITHDRAWN)])
@pytest.mark.parametrize("shape", BWD_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_rope_training(shape, dtype, pm):
    B, heads, H, W, k, s = shape
    theta, scale = 100.0, 0.5
    f32 = dtype == "f32"
    _say("rope training %s %s pad_mode=%d" % (shape, dtype, pm))
    wl = synth.Workload("case", B, heads, H, W, 64, k, s, dtype, seed=300 + sum(shape) + pm, pad_mode=pm)
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    L = H * W
    out = torch.full_like(q, float("nan"))
    lse = torch.full((B, heads, L), float("nan"), dtype=torch.float32, device="cuda")
    assert not f32
    fb.fla_swin_attn_rope_fwd_lse(q, kk, v, out, lse, B, heads, H, W, 64, k, s, pm, theta, scale)
    plain = torch.empty_like(q)
    fb.fla_swin_attn_rope_fwd(q, kk, v, plain, B, heads, H, W, 64, k, s, pm, theta, scale, f32=f32)
    dq, dk, dv = (torch.full_like(t, float("nan")) for t in (q, kk, v))
    nws = fb.fla_swin_attn_bwd_workspace(B, heads, [(H, W)], k, s, pm)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    fb.fla_swin_attn_rope_bwd(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, H, W, 64, k, s, pm, theta,
                              scale)
    torch.cuda.synchronize()
    assert torch.equal(out, plain)
    qn, kn, vn, dn = (synth.to_f64_numpy(t) for t in (q, kk, v, dout))
    lerr = np.abs(synth.to_f64_numpy(lse) - O.swin_attention_rope_lse(qn, kn, vn, H, W, k, s, pm, theta, scale))
    if f32:
        assert lerr.max() <= 1e-5, lerr.max()
    else:
        # the plain bound plus the bf16 rounding of the rotated q and k: each element moves by at
        # most 2^-9 relative, so a logit c <q', k'> by at most 2 * 2^-9 * c |q| |k| (a rotation
        # keeps norms); per query with the largest key norm of its batch entry and head
        c = 1.0 / 8.0
        qnorm = np.linalg.norm(qn, axis=-1).transpose(0, 2, 1)                  # [B, heads, L]
        kmax = np.linalg.norm(kn, axis=-1).max(axis=1)[:, :, None]               # [B, heads, 1]
        bound = 4e-3 + 2.0 * 2.0 ** -9 * c * qnorm * kmax
        assert (lerr <= bound).all(), (lerr.max(), bound.min())
    ref = O.swin_attention_rope_bwd(qn, kn, vn, dn, H, W, k, s, pm, theta, scale)
    for name, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        _check_grad(name, got, r, f32)
    if pm == 1:
        _check_grad("dk_pad", dk[:, -1], ref[1][:, -1], f32, bulk=False)

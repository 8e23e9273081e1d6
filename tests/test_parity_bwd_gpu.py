"""GPU parity of the training forward (log-sum-exp) and the backward pass against the fp64
oracle, through the C ABI.

Tolerances.  A gradient tensor has no fixed scale (dq and dk carry the factor 1/sqrt(d)),
so errors are measured against M = max |reference| of that tensor:
  * bf16: max |err| <= 2e-2 M and mean |err| <= 2e-3 M -- the forward's bf16 bounds for
    outputs of unit scale.  The kernel rounds P and dS to bf16 (relative 2^-9) before their
    products and the outputs once more; a CPU emulation of exactly these roundings on full
    16x16 windows stays below 1e-2 M (max) and 5e-4 M (mean), also with 1% of keys x8.
  * fp32: max |err| <= 1e-5 M.
  * log-sum-exp, natural log: bf16 4e-3 absolute -- the bf16 forward sums probabilities
    rounded to bf16 (relative 2^-9 each, so the sum is off by at most 2^-9 relative and its
    log by at most 2^-9 ~ 1.95e-3), twice that for margin; fp32 1e-5.
A reference that is exactly zero (one-token windows) instead needs |got| <= 1e-5.  The pad
token's gradient row (64 values per head) is checked on its own scale with the max bound only:
a mean over so few values is no bulk statistic, and when the pad token carries almost all of
a query's weight (e.g. a 1 x 40 grid with window 16: multiplicity >= 240) its dS = P (dP - D)
is a difference of nearly equal terms, where D = <dO, O> from the bf16 output dominates.
Outputs start as NaN so that an unwritten element fails."""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import swin_oracle as SO
from paper_2407_02109_amd import binding as fb
from paper_2407_02109_amd import synth

pytestmark = pytest.mark.gpu

BF16_MAX, BF16_MEAN, F32_MAX = 2e-2, 2e-3, 1e-5
LSE_BF16, LSE_F32 = 4e-3, 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fb.load_library()


def _say(msg):
    print("[case] %s" % msg, flush=True)


def _wl(B, heads, H, W, k, s, dtype, pm, seed, grids=()):
    return synth.Workload("case", B, heads, H, W, 64, k, s, dtype, seed=seed, pad_mode=pm, grids=grids)


def _train(wl, q, k, v, dout):
    """GPU training forward + backward; returns out, lse, dq, dk, dv (device tensors)."""
    B, L, heads, d = q.shape
    f32 = q.dtype == torch.float32
    out = torch.full_like(q, float("nan"))
    lse = torch.full((B, heads, L), float("nan"), dtype=torch.float32, device=q.device)
    grids = wl.grid_list
    fb.fla_swin_attn_ms_fwd_lse(q, k, v, out, lse, B, heads, grids, d, wl.window, wl.shift, wl.pad_mode,
                                f32=f32)
    dq, dk, dv = (torch.full_like(t, float("nan")) for t in (q, k, v))
    nbytes = fb.fla_swin_attn_bwd_workspace(B, heads, grids, wl.window, wl.shift, wl.pad_mode)
    ws = torch.full((max(nbytes // 4, 4),), float("nan"), dtype=torch.float32, device=q.device)
    fb.fla_swin_attn_ms_bwd(q, k, v, out, dout, lse, dq, dk, dv, ws, nbytes, B, heads, grids, d,
                            wl.window, wl.shift, wl.pad_mode, f32=f32)
    torch.cuda.synchronize()
    return out, lse, dq, dk, dv


def _check_grad(name, got, ref, f32, bulk=True):
    got = synth.to_f64_numpy(got)
    assert np.isfinite(got).all(), "%s: non-finite element (unwritten?)" % name
    M = np.abs(ref).max()
    if M < 1e-12:
        # an exactly zero gradient (a one-token window: P = 1 and dS = <dO, v> - <dO, o> = 0);
        # only fp32 rounding of the two dot products remains
        assert np.abs(got).max() <= 1e-5, (name, np.abs(got).max())
        return 0.0
    err = np.abs(got - ref)
    if f32:
        assert err.max() <= F32_MAX * M, (name, err.max() / M)
    else:
        assert err.max() <= BF16_MAX * M, (name, err.max() / M)
        if bulk:
            assert err.mean() <= BF16_MEAN * M, (name, err.mean() / M)
    return err.max() / M


SHAPES = [  # B, heads, H, W, window, shift
    (2, 2, 64, 64, 16, 8), (1, 3, 37, 29, 16, 8), (2, 2, 20, 13, 8, 3), (1, 2, 23, 41, 12, 5),
    (1, 1, 9, 7, 16, 0), (1, 2, 5, 6, 1, 0), (1, 2, 16, 16, 16, 0), (1, 2, 33, 17, 5, 2),
    (1, 1, 1, 1, 1, 0), (1, 1, 9, 300, 16, 15), (1, 2, 1, 40, 16, 7), (2, 1, 40, 1, 8, 7),
]
WIDE = [(1, 2, 40, 24, 20, 10), (1, 1, 40, 40, 32, 16), (2, 1, 37, 45, 17, 6)]   # windows over 256 tokens


def _case(B, heads, H, W, k, s, dtype, pm, seed):
    wl = _wl(B, heads, H, W, k, s, dtype, pm, seed)
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    out, lse, dq, dk, dv = _train(wl, q, kk, v, dout)
    return wl, (q, kk, v, dout), (out, lse, dq, dk, dv)


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_lse_and_backward(shape, dtype, pm):
    B, heads, H, W, k, s = shape
    _say("bwd %s %s pad_mode=%d" % (shape, dtype, pm))
    wl, ins, outs = _case(B, heads, H, W, k, s, dtype, pm, seed=100 + sum(shape) + pm)
    q, kk, v, dout = (synth.to_f64_numpy(t) for t in ins)
    out, lse, dq, dk, dv = outs
    f32 = dtype == "f32"
    # the training forward's output is the plain forward's, bit for bit, and the single-grid
    # entry point gives what the grid-list one gave
    ref_out = torch.empty_like(ins[0])
    fn = fb.fla_swin_attn_fwd_f32 if f32 else fb.fla_swin_attn_fwd
    fn(ins[0], ins[1], ins[2], ref_out, B, heads, H, W, 64, k, s, pm)
    out1 = torch.empty_like(ins[0])
    lse1 = torch.empty_like(lse)
    fb.fla_swin_attn_fwd_lse(ins[0], ins[1], ins[2], out1, lse1, B, heads, H, W, 64, k, s, pm, f32=f32)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out) and torch.equal(out1, out) and torch.equal(lse1, lse)
    lse_ref = O.swin_attention_lse(q, kk, v, H, W, k, s, pm)
    lerr = np.abs(synth.to_f64_numpy(lse) - lse_ref).max()
    assert lerr <= (LSE_F32 if f32 else LSE_BF16), lerr
    gq, gk, gv = O.swin_attention_bwd(q, kk, v, dout, H, W, k, s, pm)
    for name, got, ref in (("dq", dq, gq), ("dk", dk, gk), ("dv", dv, gv)):
        _check_grad(name, got, ref, f32)
    if pm == 1:   # the pad row on its own scale (64 values per head: the max bound only)
        _check_grad("dk_pad", dk[:, -1], gk[:, -1], f32, bulk=False)
        _check_grad("dv_pad", dv[:, -1], gv[:, -1], f32, bulk=False)


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", WIDE, ids=lambda s: "x".join(map(str, s)))
def test_backward_wide_windows(shape, dtype, pm):
    """Windows of more than 256 tokens: bf16 in 128-token blocks that each stream the whole
    window's other side through LDS in 128-token chunks (the last ones partial); fp32 in the
    three fp32 kernels."""
    B, heads, H, W, k, s = shape
    _say("bwd wide %s %s pad_mode=%d" % (shape, dtype, pm))
    f32 = dtype == "f32"
    wl, ins, outs = _case(B, heads, H, W, k, s, dtype, pm, seed=7 + pm + sum(shape))
    q, kk, v, dout = (synth.to_f64_numpy(t) for t in ins)
    _, lse, dq, dk, dv = outs
    lerr = np.abs(synth.to_f64_numpy(lse) - O.swin_attention_lse(q, kk, v, H, W, k, s, pm)).max()
    assert lerr <= (LSE_F32 if f32 else LSE_BF16), lerr
    gq, gk, gv = O.swin_attention_bwd(q, kk, v, dout, H, W, k, s, pm)
    for name, got, ref in (("dq", dq, gq), ("dk", dk, gk), ("dv", dv, gv)):
        _check_grad(name, got, ref, f32)
    if pm == 1:
        _check_grad("dk_pad", dk[:, -1], gk[:, -1], f32, bulk=False)
        _check_grad("dv_pad", dv[:, -1], gv[:, -1], f32, bulk=False)


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
def test_bf16_backward_wide_windows_multi_scale(pm):
    """A grid list whose first grid has windows of more than 256 tokens and whose second has
    small ones, in one launch."""
    grids = ((40, 37), (9, 9))
    wl = _wl(1, 2, 40, 37, 20, 10, "bf16", pm, 31 + pm, grids=grids)
    _say("bwd wide multi-scale %s pad_mode=%d" % (grids, pm))
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    _, lse, dq, dk, dv = _train(wl, q, kk, v, dout)
    qn, kn, vn, gn = (synth.to_f64_numpy(t) for t in (q, kk, v, dout))
    assert np.abs(synth.to_f64_numpy(lse) - O.swin_attention_ms_lse(qn, kn, vn, grids, 20, 10, pm)).max() <= LSE_BF16
    gq, gk, gv = O.swin_attention_ms_bwd(qn, kn, vn, gn, grids, 20, 10, pm)
    for name, got, ref in (("dq", dq, gq), ("dk", dk, gk), ("dv", dv, gv)):
        _check_grad(name, got, ref, False)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
@pytest.mark.parametrize("grids", [((40, 36), (9, 9), (3, 20)),
                                   # the most grids one launch takes (8)
                                   ((20, 13), (7, 9), (16, 16), (1, 1), (9, 30), (3, 3), (12, 5), (8, 8))],
                         ids=["3grids", "8grids"])
def test_multiscale_backward(dtype, pm, grids):
    _say("bwd ms %s %s pad_mode=%d" % (grids, dtype, pm))
    wl = _wl(2, 2, grids[0][0], grids[0][1], 16, 8, dtype, pm, 21 + pm, grids=grids)
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    _, lse, dq, dk, dv = _train(wl, q, kk, v, dout)
    qn, kn, vn, dn = (synth.to_f64_numpy(t) for t in (q, kk, v, dout))
    lerr = np.abs(synth.to_f64_numpy(lse) - O.swin_attention_ms_lse(qn, kn, vn, grids, 16, 8, pm)).max()
    assert lerr <= (LSE_F32 if dtype == "f32" else LSE_BF16)
    ref = O.swin_attention_ms_bwd(qn, kn, vn, dn, grids, 16, 8, pm)
    for name, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        _check_grad(name, got, r, dtype == "f32")


@pytest.mark.parametrize("k,s,pm", [(16, 8, 1), (20, 10, 1), (32, 16, 1)])
def test_workspace_contents_are_ignored(k, s, pm):
    """Every workspace element a call reads (the pad partials) was written by that call, and
    the result is the same bits run to run."""
    wl = _wl(1, 2, 37, 29, k, s, "bf16", pm, 5)
    _say("bwd workspace k=%d s=%d pad_mode=%d" % (k, s, pm))
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    first = _train(wl, q, kk, v, dout)   # workspace starts as NaN inside _train
    B, L, heads, d = q.shape
    nbytes = fb.fla_swin_attn_bwd_workspace(B, heads, wl.grid_list, k, s, pm)
    assert nbytes > 0
    ws = torch.full((nbytes // 4,), 1e30, dtype=torch.float32, device="cuda")
    dq, dk, dv = (torch.empty_like(t) for t in (q, kk, v))
    fb.fla_swin_attn_bwd(q, kk, v, first[0], dout, first[1], dq, dk, dv, ws, nbytes, B, heads, wl.H, wl.W,
                         d, k, s, pm)
    torch.cuda.synchronize()
    for a, b in zip((dq, dk, dv), first[2:]):
        assert torch.equal(a, b)


# ---- full size: sampled windows against the oracle, computed window by window ---------
def _window_rects(H, W, k, s):
    ry = SO._region(np.arange(H), k, s)
    rx = SO._region(np.arange(W), k, s)
    ys = [np.flatnonzero(ry == r) for r in np.unique(ry)]
    xs = [np.flatnonzero(rx == r) for r in np.unique(rx)]
    return [(y[0], y[-1] + 1, x[0], x[-1] + 1) for y in ys for x in xs]


def _window_grads(q, kk, v, dout, H, W, rect, k, pm, L):
    """Oracle gradients of one window's tokens: the window alone is a grid of one region
    (window k, no shift), and in KV-token mode keeps its pad multiplicity k^2 - n."""
    y0, y1, x0, x1 = rect
    idx = (np.arange(y0, y1)[:, None] * W + np.arange(x0, x1)[None, :]).ravel()
    rows = np.concatenate([idx, [L]]) if pm else idx
    g = O.swin_attention_bwd(q[:, idx], kk[:, rows], v[:, rows], dout[:, idx], y1 - y0, x1 - x0, k, 0, pm)
    return idx, g


FULL_SIZE = {   # the 4096^2 layer; with window 32 every window but the border ones has 1024 tokens
    "img4096": synth.WORKLOADS["img4096"],
    "img4096_kv": synth.WORKLOADS["img4096_kv"],
    "img4096_w32": synth.WORKLOADS["img4096"].with_(name="img4096_w32", window=32, shift=16),
    "img4096_kv_w32": synth.WORKLOADS["img4096_kv"].with_(name="img4096_kv_w32", window=32, shift=16),
}


@pytest.mark.parametrize("name", list(FULL_SIZE))
def test_full_size_sampled_windows(name):
    wl = FULL_SIZE[name]
    _say("bwd full size %s" % name)
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    out1 = _train(wl, q, kk, v, dout)
    out2 = _train(wl, q, kk, v, dout)
    for a, b in zip(out1, out2):
        assert torch.equal(a, b), "backward is not deterministic"
    _, lse, dq, dk, dv = (synth.to_f64_numpy(t) for t in out1)
    for t in (lse, dq, dk, dv):
        assert np.isfinite(t).all()
    qn, kn, vn, dn = (synth.to_f64_numpy(t) for t in (q, kk, v, dout))
    H, W, k, s, pm, L = wl.H, wl.W, wl.window, wl.shift, wl.pad_mode, wl.L
    rects = _window_rects(H, W, k, s)
    nwx = len(np.unique(SO._region(np.arange(W), k, s)))
    pick = sorted({0, nwx - 1, len(rects) - nwx, len(rects) - 1, 1, nwx, len(rects) // 2, 5 * nwx + 7})
    ref = {"dq": [], "dk": [], "dv": []}
    got = {"dq": [], "dk": [], "dv": []}
    for i in pick:
        idx, (gq, gk, gv) = _window_grads(qn, kn, vn, dn, H, W, rects[i], k, pm, L)
        n = len(idx)
        for key, gt, rf in (("dq", dq[:, idx], gq), ("dk", dk[:, idx], gk[:, :n]), ("dv", dv[:, idx], gv[:, :n])):
            got[key].append(gt)
            ref[key].append(rf)
    for key in ref:
        _check_grad(key, torch.from_numpy(np.concatenate(got[key], axis=1)), np.concatenate(ref[key], axis=1),
                    False)
    if pm == 1:
        # the pad row: the sum over every window with virtual slots
        pk = np.zeros_like(dk[:, L])
        pv = np.zeros_like(dv[:, L])
        for rect in rects:
            if (rect[1] - rect[0]) * (rect[3] - rect[2]) < k * k:
                idx, (_, gk, gv) = _window_grads(qn, kn, vn, dn, H, W, rect, k, pm, L)
                pk += gk[:, len(idx)]
                pv += gv[:, len(idx)]
        _check_grad("dk_pad", torch.from_numpy(dk[:, L]), pk, False, bulk=False)
        _check_grad("dv_pad", torch.from_numpy(dv[:, L]), pv, False, bulk=False)


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
def test_backward_tensors_beyond_2gib(pm):
    """Training forward and backward on 24 batch entries of the 4096^2 layer (2.4 GB per
    tensor): the last entry's windows and pad row lie past 2^31 bytes from the tensor start.
    Inputs are drawn on the GPU from a seeded generator; windows of the last entry (corner,
    border, interior) and, in KV-token mode, its pad row are checked against the oracle run on
    that entry alone."""
    B, heads, H, W, k, s = 24, 12, 256, 256, 16, 8
    L = H * W
    _say("bwd beyond 2 GiB pm=%d" % pm)
    wl = synth.Workload("big", B, heads, H, W, 64, k, s, "bf16", seed=0, pad_mode=pm)
    g = torch.Generator(device="cuda")
    g.manual_seed(21 + pm)
    rows = L + (1 if pm else 0)
    q = torch.randn(B, L, heads, 64, generator=g, device="cuda", dtype=torch.bfloat16)
    kk = torch.randn(B, rows, heads, 64, generator=g, device="cuda", dtype=torch.bfloat16)
    v = torch.randn(B, rows, heads, 64, generator=g, device="cuda", dtype=torch.bfloat16)
    dout = torch.randn(B, L, heads, 64, generator=g, device="cuda", dtype=torch.bfloat16)
    assert kk.numel() * 2 > (1 << 31)
    _, _, dq, dk, dv = _train(wl, q, kk, v, dout)
    last = slice(B - 1, B)
    qn, kn, vn, dn = (synth.to_f64_numpy(t[last]) for t in (q, kk, v, dout))
    dqn, dkn, dvn = (synth.to_f64_numpy(t[last]) for t in (dq, dk, dv))
    rects = _window_rects(H, W, k, s)
    nwx = len(np.unique(SO._region(np.arange(W), k, s)))
    pick = sorted({0, nwx - 1, len(rects) - 1, nwx + 1, len(rects) // 2})
    got = {"dq": [], "dk": [], "dv": []}
    ref = {"dq": [], "dk": [], "dv": []}
    for i in pick:
        idx, (gq, gk, gv) = _window_grads(qn, kn, vn, dn, H, W, rects[i], k, pm, L)
        n = len(idx)
        for key, gt, rf in (("dq", dqn[:, idx], gq), ("dk", dkn[:, idx], gk[:, :n]), ("dv", dvn[:, idx], gv[:, :n])):
            got[key].append(gt)
            ref[key].append(rf)
    for key in ref:
        _check_grad(key, torch.from_numpy(np.concatenate(got[key], axis=1)), np.concatenate(ref[key], axis=1),
                    False)
    if pm == 1:
        pk = np.zeros_like(dkn[:, L])
        pv = np.zeros_like(dvn[:, L])
        for rect in rects:
            if (rect[1] - rect[0]) * (rect[3] - rect[2]) < k * k:
                idx, (_, gk, gv) = _window_grads(qn, kn, vn, dn, H, W, rect, k, pm, L)
                pk += gk[:, len(idx)]
                pv += gv[:, len(idx)]
        _check_grad("dk_pad", torch.from_numpy(dkn[:, L]), pk, False, bulk=False)
        _check_grad("dv_pad", torch.from_numpy(dvn[:, L]), pv, False, bulk=False)

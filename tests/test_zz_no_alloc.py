"""The allocation-free backward (static device scratch as its workspace) against the backward
that takes the caller's workspace, through the C ABI.

Both run the same kernels on the same inputs, and the backward's summation order is fixed,
so the gradients must agree bit for bit; the first case is also held to the oracle's bounds.
Each case makes two calls in a row, the second on a smaller problem, so that the second
reads a scratch that still holds the first call's partials."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2407_02109_amd import binding as fb
from paper_2407_02109_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fb.load_library()


def _inputs(B, heads, H, W, k, s, pm, seed):
    wl = synth.Workload("noalloc", B, heads, H, W, 64, k, s, "bf16", seed=seed, pad_mode=pm)
    q, kk, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    out = torch.empty_like(q)
    lse = torch.empty((B, heads, H * W), dtype=torch.float32, device="cuda")
    fb.fla_swin_attn_fwd_lse(q, kk, v, out, lse, B, heads, H, W, 64, k, s, pm)
    return wl, q, kk, v, dout, out, lse


def _with_workspace(wl, q, kk, v, dout, out, lse):
    dq, dk, dv = (torch.full_like(t, float("nan")) for t in (q, kk, v))
    n = fb.fla_swin_attn_bwd_workspace(wl.B, wl.heads, [(wl.H, wl.W)], wl.window, wl.shift, wl.pad_mode)
    ws = torch.full((max(n // 4, 4),), float("nan"), dtype=torch.float32, device="cuda")
    fb.fla_swin_attn_bwd(q, kk, v, out, dout, lse, dq, dk, dv, ws, n, wl.B, wl.heads, wl.H, wl.W, 64,
                         wl.window, wl.shift, wl.pad_mode)
    return dq, dk, dv


def _noalloc(wl, q, kk, v, dout, out, lse):
    dq, dk, dv = (torch.full_like(t, float("nan")) for t in (q, kk, v))
    fb.fla_swin_attn_bwd_noalloc(q, kk, v, out, dout, lse, dq, dk, dv, wl.B, wl.heads, wl.H, wl.W, 64,
                                 wl.window, wl.shift, wl.pad_mode)
    return dq, dk, dv


# pairs of (B, heads, H, W, window, shift, pad_mode): the second call of a pair is smaller
PAIRS = [
    ((1, 12, 64, 64, 16, 8, 1), (2, 2, 20, 13, 8, 3, 1)),      # pad partials in the scratch
    ((1, 2, 64, 64, 32, 16, 1), (1, 1, 24, 40, 32, 16, 1)),    # windows of several blocks
    ((1, 1, 48, 64, 32, 16, 0), (2, 1, 30, 20, 16, 8, 0)),     # MASK mode: no scratch at all
]


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: "_then_".join("x".join(map(str, c)) for c in p))
def test_noalloc_matches_workspace_entry_point(pair):
    for i, case in enumerate(pair):
        print("[case] noalloc %s call %d" % (case, i + 1), flush=True)
        B, heads, H, W, k, s, pm = case
        args = _inputs(B, heads, H, W, k, s, pm, seed=40 + i)
        ref = _with_workspace(*args)
        got = _noalloc(*args)
        torch.cuda.synchronize()
        for name, g, r in zip(("dq", "dk", "dv"), got, ref):
            assert torch.isfinite(g.float()).all(), (case, name)
            assert torch.equal(g, r), (case, name, (g.float() - r.float()).abs().max().item())


def test_noalloc_against_the_oracle():
    """Two calls in a row (KV-token mode, ragged grid, then a smaller one), each within the
    backward's bf16 bounds of the fp64 oracle: max 2e-2 M, mean 2e-3 M, M = max |reference|."""
    for i, case in enumerate(((2, 3, 37, 29, 16, 8, 1), (1, 2, 9, 40, 16, 15, 1))):
        print("[case] noalloc vs oracle %s" % (case,), flush=True)
        B, heads, H, W, k, s, pm = case
        wl, q, kk, v, dout, out, lse = _inputs(B, heads, H, W, k, s, pm, seed=50 + i)
        got = _noalloc(wl, q, kk, v, dout, out, lse)
        torch.cuda.synchronize()
        refs = O.swin_attention_bwd(*(synth.to_f64_numpy(t) for t in (q, kk, v, dout)), H, W, k, s, pm)
        for name, g, r in zip(("dq", "dk", "dv"), got, refs):
            g = synth.to_f64_numpy(g)
            M = np.abs(r).max()
            e = np.abs(g - r)
            assert np.isfinite(g).all() and e.max() <= 2e-2 * M and e.mean() <= 2e-3 * M, (case, name)


def test_noalloc_rejects_problems_beyond_the_scratch():
    """A problem whose workspace exceeds the static scratch is refused, and no output is touched:
    window 1 on a 128 x 128 grid in KV-token mode has one 512-byte pad partial per token and
    head, 24 MiB for 3 heads."""
    H = W = 128
    q = torch.zeros(1, H * W, 3, 64, dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros(1, H * W + 1, 3, 64, dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros(1, 3, H * W, dtype=torch.float32, device="cuda")
    dq = torch.full_like(q, float("nan"))
    dk, dv = torch.full_like(kv, float("nan")), torch.full_like(kv, float("nan"))
    assert fb.fla_swin_attn_bwd_workspace(1, 3, [(H, W)], 1, 0, 1) == 24 << 20
    rc = fb.fla_swin_attn_bwd_noalloc(q, kv, kv, q, q, lse, dq, dk, dv, 1, 3, H, W, 64, 1, 0, 1, check=False)
    torch.cuda.synchronize()
    assert rc == 15, fb.fla_status_string(rc)
    assert all(torch.isnan(t.float()).all() for t in (dq, dk, dv))

"""GPU parity of the Cycle-scan kernels against the fp64 oracle (``oracle.cycle_scan``).

Tolerance, from the fp32 arithmetic: the kernels form Bbar = (exp(Delta a) - 1) / a * b from
the hardware exp2, whose result near 1 carries an absolute error of about 2^-24, so Bbar's
relative error is about 2^-24 / |Delta a|; the scan's other steps add a few ulps.  The bar is
max|y - y_oracle| <= (4 * 2^-24 / min|Delta a| + 1e-6) * max|y_oracle|, min over the inputs
(about 2.4e-4 for Mamba's step sizes down to 0.001 with |a| >= 1; about 1e-5 for the "wide"
inputs).  Sec. 3.5 (the SSM equations and the Cycle-scan strategy)."""
import numpy as np
import pytest
import torch

from oracle import cycle_scan as CS
from paper_2407_02109_amd import binding as fb, synth

pytestmark = pytest.mark.gpu


def _tol(delta, A):
    m = (delta.abs().amin(dim=(0, 1))[:, None] * A.abs()).min().item()
    return 4.0 * 2.0 ** -24 / m + 1e-6


def _run(x, delta, A, Bm, Cm, repeats, y=None, ws_fill=None):
    B, L, d = x.shape
    N = A.shape[1]
    dev = torch.device("cuda")
    t = [v.to(dev) for v in (x, delta, A, Bm, Cm)]
    out = torch.full((B, L, d), float("nan"), device=dev) if y is None else y
    nws = fb.fla_cycle_scan_workspace(B, L, d, N, repeats)
    ws = torch.empty(max(nws, 4) // 4, dtype=torch.float32, device=dev)
    ws.fill_(float("nan") if ws_fill is None else ws_fill)
    fb.fla_cycle_scan(*t, out, ws, ws.numel() * 4, B, L, d, N, repeats)
    torch.cuda.synchronize()
    return out.cpu()


CASES = [  # B, L, d, N, repeats
    (2, 37, 70, 4, 3),      # two chunks of 32 (the second of 5 tokens), channels past a multiple of 64
    (1, 513, 64, 32, 3),    # 32 states, 17 chunks
    (1, 3000, 96, 16, 3),   # chunks of 64 tokens
    (1, 1, 5, 1, 3),        # one token, one state
    (3, 100, 130, 8, 2),    # three batch entries, three channel groups, two copies
    (1, 257, 64, 2, 1),     # one copy: the plain scan
    (1, 700, 64, 32, 4),    # four copies
    (2, 64, 1, 4, 5),       # one channel (one live lane per wave), two whole chunks, five copies
    (1, 25600, 40, 4, 3),   # 100 chunks of 256 tokens: the carry pass in four segments
    (1, 70000, 40, 2, 2),   # 274 chunks: eight segments of two load batches each
]


@pytest.mark.parametrize("kind", ["mamba", "wide"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_cycle_scan_matches_oracle(case, kind):
    B, L, d, N, r = case
    x, delta, A, Bm, Cm = synth.make_cycle_inputs(B, L, d, N, seed=100 + L + N, kind=kind)
    y = _run(x, delta, A, Bm, Cm, r).double().numpy()
    ref = CS.cycle_scan(x.double().numpy(), delta.double().numpy(), A.double().numpy(), Bm.double().numpy(),
                        Cm.double().numpy(), r)
    assert np.isfinite(y).all()
    err = np.abs(y - ref).max() / np.abs(ref).max()
    assert err <= _tol(delta, A), (case, kind, err, _tol(delta, A))


def test_cycle_scan_full_size_sampled_channels():
    wl = synth.CYCLE_WORKLOADS["cyclescan_img4096"]
    x, delta, A, Bm, Cm = synth.make_cycle_inputs(wl.B, wl.L, wl.d, wl.N, wl.seed, wl.kind)
    y = _run(x, delta, A, Bm, Cm, wl.repeats)
    assert torch.isfinite(y).all()
    ch = [0, 1, 383, wl.d - 1]
    ref = CS.cycle_scan_channels(x.double().numpy(), delta.double().numpy(), A.double().numpy(), Bm.double().numpy(),
                                 Cm.double().numpy(), ch, wl.repeats)
    got = y[:, :, ch].double().numpy()
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err <= _tol(delta, A), err


def test_cycle_scan_is_deterministic_and_ignores_the_workspace():
    x, delta, A, Bm, Cm = synth.make_cycle_inputs(2, 1500, 130, 16, seed=7)
    a = _run(x, delta, A, Bm, Cm, 3, ws_fill=float("nan"))
    b = _run(x, delta, A, Bm, Cm, 3, ws_fill=1e30)
    assert torch.isfinite(a).all()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_cycle_scan_wrapper_and_empty_calls():
    x, delta, A, Bm, Cm = (t.cuda() for t in synth.make_cycle_inputs(1, 90, 64, 8, seed=3))
    y = fb.cycle_scan(x, delta, A, Bm, Cm, 3)
    torch.cuda.synchronize()
    ref = CS.cycle_scan(*(t.double().cpu().numpy() for t in (x, delta, A, Bm, Cm)), 3)
    assert np.abs(y.double().cpu().numpy() - ref).max() / np.abs(ref).max() <= _tol(delta.cpu(), A.cpu())
    e = torch.empty(1, 0, 64, device="cuda")
    assert fb.fla_cycle_scan(e, e, A, Bm, Cm, e, None, 0, 1, 0, 64, 8, 3) == 0
    with pytest.raises(ValueError):
        fb.cycle_scan(x, delta, A[:, :4], Bm, Cm)


def test_cycle_scan_beyond_2gib():
    """11 batch entries of the 65536-token, 768-channel sequence: x, Delta and y hold 2.2 GB each, so the last
    entries lie past 2^31 bytes from the tensors' start.  Inputs are drawn on the GPU from a seeded generator;
    sampled channels of the first and the last entry are checked against the oracle on that entry alone."""
    B, L, d, N, r = 11, 65536, 768, 32, 3
    assert B * L * d * 4 > 2 ** 31
    dev = torch.device("cuda")
    g = torch.Generator(device=dev).manual_seed(2024)
    x = torch.randn(B, L, d, device=dev, generator=g)
    delta = torch.exp(-4.0 + 2.0 * torch.rand(B, L, d, device=dev, generator=g))   # in [e^-4, e^-2]
    A = -(0.5 + 3.0 * torch.rand(d, N, device=dev, generator=g))
    Bm = torch.randn(B, L, N, device=dev, generator=g)
    Cm = torch.randn(B, L, N, device=dev, generator=g)
    y = fb.cycle_scan(x, delta, A, Bm, Cm, repeats=r)
    torch.cuda.synchronize()
    ch = [0, 767]
    tol = 4.0 * 2.0 ** -24 / (delta.amin().item() * A.abs().min().item()) + 1e-6
    for b in (0, B - 1):
        sl = lambda t: t[b:b + 1].cpu().double().numpy()
        ref = CS.cycle_scan_channels(sl(x), sl(delta), A.cpu().double().numpy(), sl(Bm), sl(Cm), ch, r)
        got = y[b:b + 1][:, :, ch].cpu().double().numpy()
        assert np.isfinite(got).all()
        err = np.abs(got - ref).max() / np.abs(ref).max()
        assert err <= tol, (b, err, tol)
    del x, delta, y
    torch.cuda.empty_cache()

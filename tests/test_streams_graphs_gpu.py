"""Launches on a non-default stream and inside captured HIP graphs (through torch.cuda.CUDAGraph,
which is a HIP graph on ROCm), compared with eager launches on the default stream.

Every entry point is asynchronous on the stream it is given and allocates nothing, so a
layer (forward, training forward, backward with its pad reduction) or a Cycle-scan call (three
kernels) can be captured once and replayed.  The graphs are replayed several times with eager work and synchronisations in
between, and every replay is checked bit for bit against the eager result."""
import pytest
import torch

from paper_2407_02109_amd import binding as fb
from paper_2407_02109_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fb.load_library()


def _say(msg):
    print("[case] %s" % msg, flush=True)


def _setup(pm):
    wl = synth.Workload("case", 2, 3, 37, 29, 64, 16, 8, "bf16", seed=77 + pm, pad_mode=pm)
    q, k, v = (t.cuda() for t in synth.make_inputs(wl))
    dout = synth.make_grad(wl).cuda()
    B, L, heads, d = q.shape
    bufs = dict(out=torch.empty_like(q), lse=torch.empty((B, heads, L), dtype=torch.float32, device="cuda"),
                dq=torch.empty_like(q), dk=torch.empty_like(k), dv=torch.empty_like(v))
    nws = fb.fla_swin_attn_bwd_workspace(B, heads, [(wl.H, wl.W)], wl.window, wl.shift, pm)
    bufs["ws"] = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    return wl, (q, k, v, dout), bufs, nws


def _layer(wl, ins, bufs, nws, stream):
    q, k, v, dout = ins
    B, L, heads, d = q.shape
    fb.fla_swin_attn_fwd_lse(q, k, v, bufs["out"], bufs["lse"], B, heads, wl.H, wl.W, d, wl.window, wl.shift,
                             wl.pad_mode, stream)
    fb.fla_swin_attn_bwd(q, k, v, bufs["out"], dout, bufs["lse"], bufs["dq"], bufs["dk"], bufs["dv"], bufs["ws"], nws,
                         B, heads, wl.H, wl.W, d, wl.window, wl.shift, wl.pad_mode, stream)


def _snapshot(bufs):
    return {k: v.clone() for k, v in bufs.items() if k != "ws"}


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
def test_side_stream_matches_default_stream(pm):
    _say("side stream pad_mode=%d" % pm)
    wl, ins, bufs, nws = _setup(pm)
    _layer(wl, ins, bufs, nws, torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = _snapshot(bufs)
    for t in bufs.values():
        t.zero_()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _layer(wl, ins, bufs, nws, side)
    side.synchronize()
    for key, r in ref.items():
        assert torch.equal(bufs[key], r), key


@pytest.mark.parametrize("pm", [0, 1], ids=["mask", "kvtoken"])
def test_graph_replays_match_eager(pm):
    _say("graph pad_mode=%d" % pm)
    wl, ins, bufs, nws = _setup(pm)
    _layer(wl, ins, bufs, nws, torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = _snapshot(bufs)
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        _layer(wl, ins, bufs, nws, cap)   # warm-up on the capture stream
    cap.synchronize()
    with torch.cuda.graph(graph, stream=cap):
        _layer(wl, ins, bufs, nws, cap)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in bufs.values():
            t.fill_(7)                      # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for key, r in ref.items():
            assert torch.equal(bufs[key], r), (rep, key)


def _cycle_setup():
    B, L, d, N, r = 2, 1500, 130, 16, 3   # several chunks, a partial channel group
    ins = [t.cuda() for t in synth.make_cycle_inputs(B, L, d, N, seed=88)]
    nws = fb.fla_cycle_scan_workspace(B, L, d, N, r)
    bufs = dict(y=torch.empty((B, L, d), dtype=torch.float32, device="cuda"),
                ws=torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda"))
    return (B, L, d, N, r), ins, bufs, nws


def _cycle(shape, ins, bufs, nws, stream):
    B, L, d, N, r = shape
    fb.fla_cycle_scan(*ins, bufs["y"], bufs["ws"], nws, B, L, d, N, r, stream)


def test_cycle_scan_side_stream_and_graph_replays_match_eager():
    _say("Cycle-scan side stream and graph")
    shape, ins, bufs, nws = _cycle_setup()
    _cycle(shape, ins, bufs, nws, torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = bufs["y"].clone()
    bufs["y"].zero_()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _cycle(shape, ins, bufs, nws, side)
    side.synchronize()
    assert torch.equal(bufs["y"], ref)
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        _cycle(shape, ins, bufs, nws, cap)
    cap.synchronize()
    with torch.cuda.graph(graph, stream=cap):
        _cycle(shape, ins, bufs, nws, cap)   # three kernels, nothing else
    torch.cuda.synchronize()
    for rep in range(3):
        for t in bufs.values():
            t.fill_(7)                       # output and workspace overwritten between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(bufs["y"], ref), rep

"""The kernels and the C ABI, built for the CPU and run against the oracle.

The sources of the fp32 and bf16 forward and backward kernels, the Cycle-scan kernels, the device header and the C ABI (launch geometry, workgroup decode, window rectangles,
workspace layout, pad-token reduction) are compiled as host C++ against a small stand-in for
the HIP runtime (tests/native/host_emu: a launch runs each block's work items as host threads
with a barrier for __syncthreads; amdgcn_host.h gives the gfx950 builtins host definitions, the
matrix-core product, the transposing LDS read, the half-wave swap, the shuffles and the ballot
exchanging their operands between the 64 lanes of a wave), with AddressSanitizer, UndefinedBehaviorSanitizer (any report aborts the
run) and exact-size buffers.  A run must stay inside every buffer and reproduce the fp64
oracle's output, log-sum-exp and gradients (fp32: to fp32 accuracy; bf16: at the GPU tests'
bounds).  No GPU is involved."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_02109_amd", "csrc")
EMU = os.path.join(ROOT, "tests", "native", "host_emu")


def _compiler():
    for cand in ("/opt/rocm/llvm/bin/clang++", shutil.which("clang++")):
        if cand and os.path.exists(cand):
            return cand
    return None


@pytest.fixture(scope="module")
def emu_binary(tmp_path_factory):
    cxx = _compiler()
    if cxx is None:
        pytest.skip("no clang++ for the host build")
    d = tmp_path_factory.mktemp("host_emu")
    src = d / "src"
    src.mkdir()
    # sources as they are (the gfx950 builtins they use come from amdgcn_host.h, force-included)
    shutil.copy(os.path.join(CSRC, "fla_swin_bwd_f32.hip"), src / "fla_swin_bwd_f32.cpp")
    shutil.copy(os.path.join(CSRC, "fla_swin_f32.hip"), src / "fla_swin_f32.cpp")
    shutil.copy(os.path.join(CSRC, "fla_cycle_scan.hip"), src / "fla_cycle_scan.cpp")
    shutil.copy(os.path.join(CSRC, "fla_swin_api.cpp"), src / "fla_swin_api.cpp")
    shutil.copy(os.path.join(CSRC, "fla_swin_internal.h"), src / "fla_swin_internal.h")
    shutil.copy(os.path.join(CSRC, "fla_cycle_scan.h"), src / "fla_cycle_scan.h")
    shutil.copy(os.path.join(CSRC, "fla_swin_device.h"), src / "fla_swin_device.h")
    # the bf16 kernels as they are, except that their intra-wave hand-off points (compiler
    # fences on the hardware, where the 64 lanes of a wave run in lockstep) become barriers over
    # the wave's lanes, which here run as separate threads
    fence = 'asm volatile("" ::: "memory");'
    for name, fences in (("fla_swin_bf16", 1), ("fla_swin_bwd_bf16_window", 1), ("fla_swin_bwd_bf16_blocks", 3)):
        text = open(os.path.join(CSRC, name + ".hip")).read()
        assert text.count(fence) == fences, name
        (src / (name + ".cpp")).write_text(text.replace(fence, "emu_wave_barrier();"))
    exe = str(d / "run")
    cmd = [cxx, "-std=c++20", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-pthread",
           "-include", os.path.join(EMU, "amdgcn_host.h"),
           "-I", EMU, "-I", str(src), "-I", os.path.join(ROOT, "include"),
           str(src / "fla_swin_bwd_f32.cpp"), str(src / "fla_swin_f32.cpp"), str(src / "fla_cycle_scan.cpp"),
           str(src / "fla_swin_bf16.cpp"), str(src / "fla_swin_bwd_bf16_window.cpp"),
           str(src / "fla_swin_bwd_bf16_blocks.cpp"),
           str(src / "fla_swin_api.cpp"),
           os.path.join(EMU, "emu.cpp"), os.path.join(EMU, "run.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    if r.returncode != 0:
        pytest.fail("host build failed:\n" + r.stderr[-4000:])
    return exe


CASES = [  # B, heads, H, W, window, shift, pad_mode
    (2, 2, 20, 13, 8, 3, 0),    # ragged grid, split windows on every border
    (1, 3, 37, 29, 16, 8, 1),   # KV-token mode: pad token, workspace and its reduction
    (1, 1, 9, 40, 16, 15, 1),   # windows of a few rows, shift next to the window size
    (1, 2, 24, 40, 32, 16, 0),  # windows of more than 256 tokens: several query blocks
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_fp32_kernels_on_the_host(emu_binary, tmp_path, case):
    B, heads, H, W, k, s, pm = case
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([emu_binary, *map(str, case), str(tmp_path)], capture_output=True, text=True, timeout=900,
                       env=env)
    assert r.returncode == 0 and "ok" in r.stdout, r.stderr[-4000:]
    L = H * W
    rows = L + (1 if pm else 0)

    def ld(name, r_):
        a = np.fromfile(str(tmp_path / (name + ".f32")), dtype=np.float32).astype(np.float64)
        return a.reshape(B, r_, heads, 64)

    q, kk, v, dout = ld("q", L), ld("k", rows), ld("v", rows), ld("dout", L)
    out = ld("out", L)
    lse = np.fromfile(str(tmp_path / "lse.f32"), dtype=np.float32).astype(np.float64).reshape(B, heads, L)
    ref_out = O.swin_attention_textbook(q, kk, v, H, W, k, s, pm)
    ref_lse = O.swin_attention_lse(q, kk, v, H, W, k, s, pm)
    assert np.abs(out - ref_out).max() <= 1e-5
    assert np.abs(lse - ref_lse).max() <= 1e-5
    refs = O.swin_attention_bwd(q, kk, v, dout, H, W, k, s, pm)
    for name, got, ref in zip(("dq", "dk", "dv"), (ld("dq", L), ld("dk", rows), ld("dv", rows)), refs):
        m = max(1.0, np.abs(ref).max())
        assert np.abs(got - ref).max() <= 2e-5 * m, name


CYCLE_CASES = [  # B, L, d, N, repeats
    (2, 37, 70, 4, 3),     # two chunks (the second of 5 tokens), channels past a multiple of 64
    (1, 200, 64, 32, 3),   # 32 states, seven chunks
    (1, 65, 5, 1, 2),      # one state, three chunks, two copies
    (2, 33, 3, 16, 1),     # one copy: the plain scan
    (1, 3000, 8, 8, 4),    # chunks of 64 tokens, four copies
    (2, 64, 1, 4, 5),      # one channel, two whole chunks, five copies
    # the carry pass in 2, 4 and 8 segments of chunks (36, 100 and 157 chunks of 256 tokens)
    (1, 9000, 3, 4, 2),
    (1, 25600, 1, 1, 3),
    (1, 40000, 1, 2, 3),
    (1, 70000, 1, 1, 2),   # 274 chunks: 8 segments of 35, two load batches each (the second run reloads)
]


@pytest.mark.parametrize("case", CYCLE_CASES, ids=lambda c: "x".join(map(str, c)))
def test_cycle_scan_kernels_on_the_host(emu_binary, tmp_path, case):
    """The Cycle-scan kernels (their unmodified source, built for the host with
    AddressSanitizer on exact-size buffers) against the oracle's definition."""
    from oracle import cycle_scan as CS
    B, L, d, N, r = case
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    res = subprocess.run([emu_binary, "cycle", *map(str, case), str(tmp_path)], capture_output=True, text=True,
                         timeout=900, env=env)
    assert res.returncode == 0 and "ok" in res.stdout, res.stderr[-4000:]
    ld = lambda name, shape: np.fromfile(str(tmp_path / (name + ".f32")), dtype=np.float32).astype(np.float64).reshape(shape)
    x, delta, y = ld("x", (B, L, d)), ld("delta", (B, L, d)), ld("y", (B, L, d))
    A, Bm, Cm = ld("A", (d, N)), ld("Bm", (B, L, N)), ld("Cm", (B, L, N))
    ref = CS.cycle_scan(x, delta, A, Bm, Cm, r)
    err = np.abs(y - ref).max() / max(1.0, np.abs(ref).max())
    assert err <= 1e-4, err



def test_launch_failure_is_reported_and_leaves_outputs_untouched(emu_binary):
    """FLA_ERR_LAUNCH: a launch that the runtime refuses (bf16 entry points, whose launchers this
    build stubs out as failing, and the fp32 and Cycle-scan entry points with the emulated runtime
    failing every launch) returns that status and leaves out, lse, dq, dk, dv, y and the workspace
    as they were."""
    r = subprocess.run([emu_binary, "launchfail"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-2000:] + r.stderr[-4000:]


BF16_CASES = [  # kind, B, heads, grids, window, shift, pad_mode, head_dim, rope theta, rope scale
    ("plain", 1, 2, "20x13", 8, 3, 0, 64, 0, 0),
    ("plain", 1, 2, "20x13", 8, 3, 1, 64, 0, 0),     # KV-token mode: the pad token as key n
    ("plain", 2, 1, "9x40", 16, 15, 1, 64, 0, 0),    # windows of a few rows, two batch entries
    ("plain", 1, 1, "24x40", 32, 16, 0, 64, 0, 0),   # windows of up to 1024 tokens: query blocks, key chunks
    ("plain", 1, 2, "17x11", 8, 4, 1, 32, 0, 0),     # head_dim 32
    ("plain", 1, 1, "17x11", 8, 4, 0, 128, 0, 0),    # head_dim 128
    ("rope", 1, 2, "20x13", 8, 3, 1, 64, 100.0, 0.5),      # the per-window cos / sin table
    ("rope", 1, 1, "40x24", 40, 0, 0, 64, 10000.0, 1.0),   # a window wider than the table: per piece
    ("ms", 1, 2, "20x13,7x9", 8, 4, 1, 64, 0, 0),
    ("ms", 1, 1, "20x13,7x9,16x16,1x1,9x30,3x3,12x5,8x8", 8, 4, 1, 64, 0, 0),   # the most grids a launch takes
]


@pytest.mark.parametrize("case", BF16_CASES, ids=lambda c: "%s-%s-%d-%d-%d-d%d" % (c[0], c[3].replace(",", "+"), c[4],
                                                                                  c[5], c[6], c[7]))
def test_bf16_forward_on_the_host(emu_binary, tmp_path, case):
    """The bf16 forward kernel (its source, with the matrix-core products, the half-wave swap
    and the ballot emulated per wave) and the device header, built for the host with
    AddressSanitizer and UndefinedBehaviorSanitizer on exact-size buffers, against the fp64
    oracle at the GPU tests' bf16 bounds (max 2e-2, mean 2e-3)."""
    kind, B, heads, grids, k, s, pm, d, theta, scale = case
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([emu_binary, "bf16", kind, str(B), str(heads), grids, str(k), str(s), str(pm), str(d),
                        str(theta), str(scale), str(tmp_path)], capture_output=True, text=True, timeout=900, env=env)
    assert r.returncode == 0 and "ok" in r.stdout, r.stderr[-4000:]
    glist = [tuple(int(x) for x in g.split("x")) for g in grids.split(",")]
    L = sum(h * w for h, w in glist)
    rows = L + (1 if pm else 0)

    def ld(name, r_):
        u = np.fromfile(str(tmp_path / (name + ".bf16")), dtype=np.uint16).astype(np.uint32) << 16
        return u.view(np.float32).astype(np.float64).reshape(B, r_, heads, d)

    q, kk, v, out = ld("q", L), ld("k", rows), ld("v", rows), ld("out", L)
    assert np.isfinite(out).all(), "unwritten output rows"
    if kind == "plain":
        ref = O.swin_attention_textbook(q, kk, v, glist[0][0], glist[0][1], k, s, pm)
    elif kind == "rope":
        ref = O.swin_attention_rope(q, kk, v, glist[0][0], glist[0][1], k, s, pm, theta, scale)
    else:
        ref = O.swin_attention_ms(q, kk, v, glist, k, s, pm)
    err = np.abs(out - ref)
    assert err.max() <= 2e-2 and err.mean() <= 2e-3, (err.max(), err.mean())


BF16_TRAIN_CASES = [  # kind, B, heads, grids, window, shift, pad_mode, rope theta, rope scale
    ("plain", 1, 1, "13x11", 8, 3, 0, 0, 0),      # one-window kernel
    ("plain", 2, 1, "13x11", 8, 3, 1, 0, 0),      # one-window kernel, pad token, its gradient's reduction
    ("plain", 1, 1, "24x20", 20, 10, 0, 0, 0),    # windows of up to 400 tokens: key- and query-role blocks
    ("plain", 1, 1, "24x20", 20, 10, 1, 0, 0),    # the same with the pad token
    ("rope", 1, 1, "13x11", 8, 3, 1, 100.0, 0.5),
    ("rope", 1, 1, "24x20", 20, 10, 1, 100.0, 0.5),   # the block kernel's RoPE + pad instance (spills to scratch)
    ("rope", 1, 1, "33x12", 33, 0, 0, 10000.0, 1.0),  # a window taller than the forward's cos / sin table
    ("ms", 1, 1, "20x13,7x9,3x20", 8, 4, 1, 0, 0),
]


@pytest.mark.parametrize("case", BF16_TRAIN_CASES, ids=lambda c: "%s-%s-%d-%d-%d" % (c[0], c[3].replace(",", "+"),
                                                                                     c[4], c[5], c[6]))
def test_bf16_training_on_the_host(emu_binary, tmp_path, case):
    """The bf16 training forward and backward (one-window and block kernels, the pad-gradient
    reduction) on the host emulation with AddressSanitizer and UndefinedBehaviorSanitizer,
    against the fp64 oracle's gradients at the GPU tests' bounds (max 2e-2, mean 2e-3 of the
    largest reference gradient) and its log-sum-exp.  For the plain cases the driver also runs
    the allocation-free backward twice and requires the same bits as the workspace call."""
    kind, B, heads, grids, k, s, pm, theta, scale = case
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([emu_binary, "bf16train", kind, str(B), str(heads), grids, str(k), str(s), str(pm),
                        str(theta), str(scale), str(tmp_path)], capture_output=True, text=True, timeout=1200, env=env)
    assert r.returncode == 0 and "ok" in r.stdout, r.stderr[-4000:]
    glist = [tuple(int(x) for x in g.split("x")) for g in grids.split(",")]
    L = sum(h * w for h, w in glist)
    rows = L + (1 if pm else 0)

    def ld(name, r_):
        u = np.fromfile(str(tmp_path / (name + ".bf16")), dtype=np.uint16).astype(np.uint32) << 16
        return u.view(np.float32).astype(np.float64).reshape(B, r_, heads, 64)

    q, kk, v, dout = ld("q", L), ld("k", rows), ld("v", rows), ld("dout", L)
    lse = np.fromfile(str(tmp_path / "lse.f32"), dtype=np.float32).astype(np.float64).reshape(B, heads, L)
    H, W = glist[0]
    if kind == "plain":
        refs = O.swin_attention_bwd(q, kk, v, dout, H, W, k, s, pm)
        ref_lse = O.swin_attention_lse(q, kk, v, H, W, k, s, pm)
    elif kind == "rope":
        refs = O.swin_attention_rope_bwd(q, kk, v, dout, H, W, k, s, pm, theta, scale)
        ref_lse = O.swin_attention_rope_lse(q, kk, v, H, W, k, s, pm, theta, scale)
    else:
        refs = O.swin_attention_ms_bwd(q, kk, v, dout, glist, k, s, pm)
        ref_lse = O.swin_attention_ms_lse(q, kk, v, glist, k, s, pm)
    # the log-sum-exp: the forward's bound, plus for RoPE the bf16 rounding of the rotated q, k
    # (2 * 2^-9 relative per logit: a rotation keeps norms)
    bound = 4e-3
    if kind == "rope":
        qn = np.linalg.norm(q, axis=-1).transpose(0, 2, 1)
        kmax = np.linalg.norm(kk, axis=-1).max(axis=1)[:, :, None]
        bound = 4e-3 + 2.0 * 2.0 ** -9 * 0.125 * qn * kmax
    assert (np.abs(lse - ref_lse) <= bound).all()
    for name, got, ref in zip(("dq", "dk", "dv"), (ld("dq", L), ld("dk", rows), ld("dv", rows)), refs):
        assert np.isfinite(got).all(), name
        M = np.abs(ref).max()
        err = np.abs(got - ref)
        assert err.max() <= 2e-2 * M and err.mean() <= 2e-3 * M, (name, err.max() / M, err.mean() / M)

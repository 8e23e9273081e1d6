"""CPU tests of the C ABI: exported symbols, argument checks, work counts.

No kernel is launched here: every call either fails an argument check before any device
access, or (with no GPU present) stops at the architecture probe."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle as O
from paper_2407_02109_amd import binding as fb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fla_swin.h")


def _header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fla_\w+)\s*\(", text)))


def _header_enum(name):
    text = open(HEADER).read()
    return {k: int(v) for k, v in re.findall(r"\b(%s_\w+)\s*=\s*(\d+)" % name, text)}


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fb.library_path()):
        pytest.skip("libfla_swin.so not built")
    return fb.load_library()


def test_header_declares_the_entry_points():
    assert _header_functions() == sorted([
        "fla_status_string", "fla_swin_attn_fwd", "fla_swin_attn_fwd_f32", "fla_swin_attn_ms_fwd",
        "fla_swin_attn_ms_fwd_f32", "fla_swin_attn_ms_work", "fla_swin_attn_work",
        "fla_swin_attn_fwd_lse", "fla_swin_attn_fwd_lse_f32", "fla_swin_attn_ms_fwd_lse",
        "fla_swin_attn_ms_fwd_lse_f32", "fla_swin_attn_bwd_workspace", "fla_swin_attn_bwd",
        "fla_swin_attn_bwd_f32", "fla_swin_attn_ms_bwd", "fla_swin_attn_ms_bwd_f32",
        "fla_swin_attn_bwd_work", "fla_swin_attn_rope_fwd", "fla_swin_attn_rope_fwd_f32",
        "fla_swin_attn_rope_fwd_lse", "fla_swin_attn_rope_bwd", "fla_swin_attn_bwd_noalloc",
        "fla_cycle_scan", "fla_cycle_scan_workspace", "fla_cycle_scan_work"])


def test_library_exports_every_header_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", fb.library_path()],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s+(\w+)", out))
    for name in _header_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None
    # nothing else with the library prefix leaks out
    assert {s for s in exported if s.startswith("fla_")} == set(_header_functions())


def test_status_strings_cover_every_code(lib):
    codes = _header_enum("FLA")
    st = {k: v for k, v in codes.items() if k.startswith("FLA_ERR") or k == "FLA_OK"}
    assert sorted(st.values()) == list(range(len(st)))
    seen = set()
    for name, code in st.items():
        s = fb.fla_status_string(code)
        assert s and s != "unknown status", name
        seen.add(s)
    assert len(seen) == len(st)
    assert fb.fla_status_string(999) == "unknown status"
    assert fb.fla_status_string(-1) == "unknown status"


def test_status_values_are_the_interface_table():
    """The numeric status values of the interface (the ten of the boundary's contract, then the
    library's own additions after FLA_ERR_LAUNCH), and the numbers the binding exposes."""
    want = {"FLA_OK": 0, "FLA_ERR_NULL": 1, "FLA_ERR_ALIGN": 2, "FLA_ERR_SHAPE": 3, "FLA_ERR_HEAD_DIM": 4,
            "FLA_ERR_WINDOW": 5, "FLA_ERR_SHIFT": 6, "FLA_ERR_PAD_MODE": 7, "FLA_ERR_ALIAS": 8,
            "FLA_ERR_ARCH": 9, "FLA_ERR_LAUNCH": 10, "FLA_ERR_TOO_LARGE": 11, "FLA_ERR_UNSUPPORTED": 12,
            "FLA_ERR_WORKSPACE": 13, "FLA_ERR_ROPE": 14, "FLA_ERR_SCRATCH": 15}
    codes = _header_enum("FLA")
    assert {k: v for k, v in codes.items() if k.startswith("FLA_ERR") or k == "FLA_OK"} == want
    assert codes["FLA_PAD_MASK"] == 0 and codes["FLA_PAD_KVTOKEN"] == 1


def test_stream_parameter_is_a_hip_stream():
    """Every launching entry point takes its stream as hipStream_t (NULL = the null stream)."""
    text = open(HEADER).read()
    assert "void* stream" not in text
    decls = re.findall(r"int\s+(fla_swin_attn_\w+)\(([^;]*)\);", text)
    launching = [n for n, a in decls if "stream" in a]
    assert len(launching) >= 14
    for n, a in decls:
        if "stream" in a:
            assert re.search(r"hipStream_t\s+stream\s*$", a.strip()), n


# fake, 256-byte aligned, non-overlapping device addresses: never dereferenced on failure
Q, K, V, OUT = 0x10000000, 0x20000000, 0x30000000, 0x40000000
GOOD = dict(B=1, heads=12, Hgrid=64, Wgrid=64, head_dim=64, window=16, shift=8, pad_mode=0)


def _call(fn, q=Q, k=K, v=V, out=OUT, **kw):
    a = dict(GOOD)
    a.update(kw)
    return fn(q, k, v, out, a["B"], a["heads"], a["Hgrid"], a["Wgrid"], a["head_dim"],
              a["window"], a["shift"], a["pad_mode"], 0, check=False)


CASES = [
    ("FLA_ERR_SHAPE", dict(B=-1)), ("FLA_ERR_SHAPE", dict(heads=-3)),
    ("FLA_ERR_SHAPE", dict(Hgrid=-1)), ("FLA_ERR_SHAPE", dict(Wgrid=-64)),
    ("FLA_ERR_NULL", dict(q=0)), ("FLA_ERR_NULL", dict(k=0)), ("FLA_ERR_NULL", dict(v=0)),
    ("FLA_ERR_NULL", dict(out=0)),
    ("FLA_ERR_ALIGN", dict(q=Q + 8)), ("FLA_ERR_ALIGN", dict(out=OUT + 2)),
    ("FLA_ERR_ALIGN", dict(v=V + 4)), ("FLA_ERR_ALIGN", dict(k=K + 1)),
    ("FLA_ERR_HEAD_DIM", dict(head_dim=48)), ("FLA_ERR_HEAD_DIM", dict(head_dim=0)),
    ("FLA_ERR_HEAD_DIM", dict(head_dim=16)), ("FLA_ERR_HEAD_DIM", dict(head_dim=256)),
    ("FLA_ERR_WINDOW", dict(window=0)), ("FLA_ERR_WINDOW", dict(window=-4, shift=0)),
    ("FLA_ERR_SHIFT", dict(shift=16)), ("FLA_ERR_SHIFT", dict(shift=-1)),
    ("FLA_ERR_SHIFT", dict(window=1, shift=1)),
    ("FLA_ERR_PAD_MODE", dict(pad_mode=2)), ("FLA_ERR_PAD_MODE", dict(pad_mode=-1)),
    ("FLA_ERR_TOO_LARGE", dict(Hgrid=1 << 20, Wgrid=1 << 20)),
    ("FLA_ERR_TOO_LARGE", dict(B=1 << 20, Hgrid=1024, Wgrid=1024)),
    ("FLA_ERR_TOO_LARGE", dict(B=2**31 - 1, heads=2**31 - 1, Hgrid=2**31 - 1, Wgrid=2**31 - 1)),
    ("FLA_ERR_TOO_LARGE", dict(Hgrid=4, Wgrid=1 << 21, window=8, shift=0)),   # window rows span 3 GiB
    ("FLA_ERR_TOO_LARGE", dict(heads=1, Hgrid=2048, Wgrid=2048, window=2048, shift=0)),  # n*cols = 2^33
    ("FLA_ERR_ALIAS", dict(out=Q)), ("FLA_ERR_ALIAS", dict(out=Q + 64 * 64 * 12 * 64)),
    ("FLA_ERR_ALIAS", dict(out=K - 256)), ("FLA_ERR_ALIAS", dict(out=V + 1024)),
]


@pytest.mark.parametrize("fn", [fb.fla_swin_attn_fwd, fb.fla_swin_attn_fwd_f32], ids=["bf16", "f32"])
@pytest.mark.parametrize("status,kw", CASES, ids=["%s-%d" % (c[0], i) for i, c in enumerate(CASES)])
def test_argument_checks(lib, fn, status, kw):
    codes = _header_enum("FLA")
    kw = dict(kw)
    if fn is fb.fla_swin_attn_fwd_f32 and status == "FLA_ERR_ALIAS" and kw.get("out") == Q + 64 * 64 * 12 * 64:
        kw["out"] = Q + 64 * 64 * 12 * 64 * 2      # still inside q: fp32 elements are 4 bytes
    assert _call(fn, **kw) == codes[status]


def test_first_failing_check_wins(lib):
    codes = _header_enum("FLA")
    # NULL and bad shift: NULL is reported (the header's check order)
    assert _call(fb.fla_swin_attn_fwd, q=0, shift=99) == codes["FLA_ERR_NULL"]
    # bad head_dim and bad shift: head_dim first
    assert _call(fb.fla_swin_attn_fwd, head_dim=48, shift=99) == codes["FLA_ERR_HEAD_DIM"]
    # negative size beats everything
    assert _call(fb.fla_swin_attn_fwd, B=-1, q=0, head_dim=1) == codes["FLA_ERR_SHAPE"]


def test_adjacent_buffers_do_not_alias(lib):
    n = 1 * 64 * 64 * 12 * 64 * 2
    st = _call(fb.fla_swin_attn_fwd, q=Q, k=Q + n, v=Q + 2 * n, out=Q + 3 * n)
    assert st != _header_enum("FLA")["FLA_ERR_ALIAS"]


@pytest.mark.parametrize("kw", [dict(B=0), dict(heads=0), dict(Hgrid=0), dict(Wgrid=0, q=0, out=0)])
def test_empty_problem_is_ok_and_ignores_pointers(lib, kw):
    kw = dict(kw)
    kw.setdefault("q", 0)
    assert _call(fb.fla_swin_attn_fwd, **kw) == 0
    assert _call(fb.fla_swin_attn_fwd_f32, **kw) == 0


def test_kvtoken_alias_range_includes_pad_row(lib):
    codes = _header_enum("FLA")
    L = 64 * 64
    tok = 12 * 64 * 2
    # k occupies L+1 rows in KV-token mode: out starting right after L rows of k overlaps
    assert _call(fb.fla_swin_attn_fwd, k=K, out=K + L * tok, pad_mode=1) == codes["FLA_ERR_ALIAS"]
    assert _call(fb.fla_swin_attn_fwd, k=K, out=K + L * tok, pad_mode=0) != codes["FLA_ERR_ALIAS"]


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
def test_no_device_reports_arch(lib):
    assert _call(fb.fla_swin_attn_fwd) == _header_enum("FLA")["FLA_ERR_ARCH"]
    assert _call(fb.fla_swin_attn_fwd_f32) == _header_enum("FLA")["FLA_ERR_ARCH"]


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
@pytest.mark.parametrize("d", [32, 128])
def test_plain_forwards_take_head_dim_32_and_128(lib, d):
    """The plain forwards (bf16 and fp32, one grid or several) pass every argument check with
    head_dim 32 or 128 (here: FLA_ERR_ARCH, the last check, on a host without the GPU); the
    training forward, RoPE and the backward take 64 only."""
    codes = _header_enum("FLA")
    assert _call(fb.fla_swin_attn_fwd, head_dim=d) == codes["FLA_ERR_ARCH"]
    assert _call(fb.fla_swin_attn_fwd_f32, head_dim=d) == codes["FLA_ERR_ARCH"]
    assert _call_ms(fb.fla_swin_attn_ms_fwd, head_dim=d) == codes["FLA_ERR_ARCH"]
    assert _call_ms(fb.fla_swin_attn_ms_fwd_f32, head_dim=d) == codes["FLA_ERR_ARCH"]
    assert _call_lse(head_dim=d) == codes["FLA_ERR_HEAD_DIM"]
    assert _call_lse(f32=True, head_dim=d) == codes["FLA_ERR_HEAD_DIM"]
    assert _call_bwd(head_dim=d) == codes["FLA_ERR_HEAD_DIM"]
    assert _call_rope(head_dim=d) == codes["FLA_ERR_HEAD_DIM"]
    assert _call_rope(f32=True, head_dim=d) == codes["FLA_ERR_HEAD_DIM"]


@pytest.mark.parametrize("B,heads,H,W,k,s,pm", [
    (1, 12, 64, 64, 16, 8, 0), (1, 12, 256, 256, 16, 8, 0), (4, 12, 150, 203, 16, 8, 0),
    (1, 1, 32, 32, 8, 4, 0), (1, 1, 32, 32, 8, 0, 0), (2, 3, 20, 13, 8, 4, 1),
    (1, 2, 7, 5, 16, 3, 1), (1, 1, 1, 1, 1, 0, 1), (3, 2, 40, 24, 64, 0, 0), (1, 12, 64, 64, 32, 16, 1)])
def test_work_counts_match_oracle(lib, B, heads, H, W, k, s, pm):
    for eb in (2, 4):
        f, b = fb.fla_swin_attn_work(B, heads, H, W, 64, k, s, pm, eb)
        f0, b0 = O.work_counts(B, heads, H, W, 64, k, s, pm, eb)
        assert f == f0 and b == b0


def test_work_counts_errors(lib):
    assert lib.fla_swin_attn_work(1, 1, 8, 8, 64, 0, 0, 0, 2, None, None) == _header_enum("FLA")["FLA_ERR_WINDOW"]
    assert lib.fla_swin_attn_work(1, 1, 8, 8, 64, 4, 4, 0, 2, None, None) == _header_enum("FLA")["FLA_ERR_SHIFT"]
    assert lib.fla_swin_attn_work(-1, 1, 8, 8, 64, 4, 0, 0, 2, None, None) == _header_enum("FLA")["FLA_ERR_SHAPE"]
    f = ctypes.c_double(-1)
    assert lib.fla_swin_attn_work(0, 1, 8, 8, 64, 4, 0, 0, 2, ctypes.byref(f), None) == 0
    assert f.value == 0.0


# ---- multi-scale entry points --------------------------------------------------------
MS_GOOD = dict(B=1, heads=12, grids=[(64, 64), (32, 32)], head_dim=64, window=16, shift=8, pad_mode=0)


def _call_ms(fn, q=Q, k=K, v=V, out=OUT, **kw):
    a = dict(MS_GOOD)
    a.update(kw)
    return fn(q, k, v, out, a["B"], a["heads"], a["grids"], a["head_dim"], a["window"], a["shift"],
              a["pad_mode"], 0, check=False)


MS_CASES = [
    ("FLA_ERR_SHAPE", dict(grids=[])), ("FLA_ERR_SHAPE", dict(grids=[(4, 4)] * 9)),
    ("FLA_ERR_SHAPE", dict(grids=[(64, 64), (-1, 32)])), ("FLA_ERR_SHAPE", dict(B=-1)),
    ("FLA_ERR_NULL", dict(q=0)), ("FLA_ERR_ALIGN", dict(out=OUT + 4)),
    ("FLA_ERR_HEAD_DIM", dict(head_dim=96)), ("FLA_ERR_SHIFT", dict(shift=16)),
    ("FLA_ERR_PAD_MODE", dict(pad_mode=3)),
    ("FLA_ERR_TOO_LARGE", dict(grids=[(64, 64), (4, 1 << 21)], window=8, shift=0)),
    ("FLA_ERR_ALIAS", dict(out=Q + (64 * 64 + 32 * 32 - 1) * 12 * 64 * 2)),   # last row of q
]


@pytest.mark.parametrize("fn", [fb.fla_swin_attn_ms_fwd, fb.fla_swin_attn_ms_fwd_f32], ids=["bf16", "f32"])
@pytest.mark.parametrize("status,kw", MS_CASES, ids=["%s-%d" % (c[0], i) for i, c in enumerate(MS_CASES)])
def test_ms_argument_checks(lib, fn, status, kw):
    kw = dict(kw)
    if fn is fb.fla_swin_attn_ms_fwd_f32 and status == "FLA_ERR_ALIAS":
        kw["out"] = Q + (64 * 64 + 32 * 32 - 1) * 12 * 64 * 4
    assert _call_ms(fn, **kw) == _header_enum("FLA")[status]


def test_ms_null_grid_list_and_empty_grids(lib):
    codes = _header_enum("FLA")
    assert lib.fla_swin_attn_ms_fwd(Q, K, V, OUT, 1, 12, 2, None, 64, 16, 8, 0, None) == codes["FLA_ERR_NULL"]
    # a grid count outside 1..8 is reported before the NULL list
    assert lib.fla_swin_attn_ms_fwd(Q, K, V, OUT, 1, 12, 0, None, 64, 16, 8, 0, None) == codes["FLA_ERR_SHAPE"]
    # every grid empty: nothing to do, pointers ignored
    assert _call_ms(fb.fla_swin_attn_ms_fwd, q=0, grids=[(0, 5), (7, 0)]) == 0


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
def test_ms_no_device_reports_arch(lib):
    assert _call_ms(fb.fla_swin_attn_ms_fwd) == _header_enum("FLA")["FLA_ERR_ARCH"]
    assert _call_ms(fb.fla_swin_attn_ms_fwd, grids=[(64, 64)]) == _header_enum("FLA")["FLA_ERR_ARCH"]


@pytest.mark.parametrize("grids,k,s,pm", [
    ([(128, 128), (32, 32)], 16, 8, 1), ([(64, 64), (32, 32)], 16, 8, 0), ([(20, 13), (7, 9), (1, 1)], 8, 3, 1),
    ([(150, 203)], 16, 8, 0), ([(5, 0), (9, 9)], 4, 1, 1)])
def test_ms_work_counts_match_oracle(lib, grids, k, s, pm):
    for eb in (2, 4):
        f, b = fb.fla_swin_attn_ms_work(2, 3, grids, 64, k, s, pm, eb)
        f0, b0 = O.ms_work_counts(2, 3, [g for g in grids if g[0] * g[1] > 0], 64, k, s, pm, eb)
        assert f == f0 and b == b0


def test_single_grid_work_equals_ms_work(lib):
    for args in [(1, 12, 256, 256, 64, 16, 8, 0, 2), (4, 12, 150, 203, 64, 16, 8, 1, 2)]:
        B, heads, H, W, d, k, s, pm, eb = args
        assert fb.fla_swin_attn_work(*args) == fb.fla_swin_attn_ms_work(B, heads, [(H, W)], d, k, s, pm, eb)


def test_product_code_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2407_02109_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "import oracle" not in text and "from oracle" not in text, fn
                assert "swin_oracle" not in text, fn


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(fb, "_lib", None)
    monkeypatch.setattr(fb, "library_path", lambda: str(tmp_path / "libfla_swin.so"))
    with pytest.raises(fb.FlaError):
        fb.load_library()


# ---- training forward and backward entry points -------------------------------------
LSE, DOUT, DQ, DK, DV, WS = 0x50000000, 0x60000000, 0x70000000, 0x80000000, 0x90000000, 0xA0000000


def _call_lse(f32=False, lse=LSE, **kw):
    a = dict(GOOD)
    a.update({k: v for k, v in kw.items() if k in GOOD})
    ptrs = dict(q=Q, k=K, v=V, out=OUT)
    ptrs.update({k: v for k, v in kw.items() if k in ptrs})
    return fb.fla_swin_attn_fwd_lse(ptrs["q"], ptrs["k"], ptrs["v"], ptrs["out"], lse, a["B"], a["heads"],
                                    a["Hgrid"], a["Wgrid"], a["head_dim"], a["window"], a["shift"],
                                    a["pad_mode"], 0, check=False, f32=f32)


def _call_bwd(f32=False, ws_bytes=1 << 24, **kw):
    a = dict(GOOD)
    a.update({k: v for k, v in kw.items() if k in GOOD})
    p = dict(q=Q, k=K, v=V, out=OUT, dout=DOUT, lse=LSE, dq=DQ, dk=DK, dv=DV, ws=WS)
    p.update({k: v for k, v in kw.items() if k in p})
    return fb.fla_swin_attn_bwd(p["q"], p["k"], p["v"], p["out"], p["dout"], p["lse"], p["dq"], p["dk"],
                                p["dv"], p["ws"], ws_bytes, a["B"], a["heads"], a["Hgrid"], a["Wgrid"],
                                a["head_dim"], a["window"], a["shift"], a["pad_mode"], 0, check=False,
                                f32=f32)


LSE_CASES = [
    ("FLA_ERR_NULL", dict(lse=0)), ("FLA_ERR_NULL", dict(q=0)), ("FLA_ERR_ALIGN", dict(lse=LSE + 4)),
    ("FLA_ERR_SHIFT", dict(shift=20)),
    ("FLA_ERR_ALIAS", dict(lse=OUT + 64)), ("FLA_ERR_ALIAS", dict(lse=Q)),
    ("FLA_ERR_ALIAS", dict(lse=K - 64 * 64 * 12 * 4 + 16)),   # lse's last bytes run into k
]


@pytest.mark.parametrize("f32", [False, True], ids=["bf16", "f32"])
@pytest.mark.parametrize("status,kw", LSE_CASES, ids=["%s-%d" % (c[0], i) for i, c in enumerate(LSE_CASES)])
def test_lse_argument_checks(lib, f32, status, kw):
    assert _call_lse(f32=f32, **kw) == _header_enum("FLA")[status]


TOK_B = 64 * 64 * 12 * 64 * 2      # bytes of one bf16 tensor of GOOD
BWD_CASES = [
    ("FLA_ERR_SHAPE", dict(B=-1)),
    ("FLA_ERR_NULL", dict(out=0)), ("FLA_ERR_NULL", dict(dout=0)), ("FLA_ERR_NULL", dict(lse=0)),
    ("FLA_ERR_NULL", dict(dq=0)), ("FLA_ERR_NULL", dict(dk=0)), ("FLA_ERR_NULL", dict(dv=0)),
    ("FLA_ERR_ALIGN", dict(dout=DOUT + 2)), ("FLA_ERR_ALIGN", dict(dv=DV + 8)),
    ("FLA_ERR_ALIGN", dict(ws=WS + 4)), ("FLA_ERR_ALIGN", dict(lse=LSE + 4)),
    ("FLA_ERR_HEAD_DIM", dict(head_dim=128)), ("FLA_ERR_WINDOW", dict(window=0)),
    ("FLA_ERR_SHIFT", dict(shift=16)), ("FLA_ERR_PAD_MODE", dict(pad_mode=5)),
    ("FLA_ERR_TOO_LARGE", dict(Hgrid=1 << 20, Wgrid=1 << 20)),
    ("FLA_ERR_WORKSPACE", dict(pad_mode=1, ws=0)), ("FLA_ERR_WORKSPACE", dict(pad_mode=1, ws_bytes=16)),
    ("FLA_ERR_ALIAS", dict(dq=Q)), ("FLA_ERR_ALIAS", dict(dk=DOUT + 128)), ("FLA_ERR_ALIAS", dict(dv=LSE)),
    ("FLA_ERR_ALIAS", dict(dv=DK + 64)), ("FLA_ERR_ALIAS", dict(pad_mode=1, ws=DQ + TOK_B - 16)),
    ("FLA_ERR_ALIAS", dict(dq=OUT + TOK_B - 16)),
]


@pytest.mark.parametrize("f32", [False, True], ids=["bf16", "f32"])
@pytest.mark.parametrize("status,kw", BWD_CASES, ids=["%s-%d" % (c[0], i) for i, c in enumerate(BWD_CASES)])
def test_bwd_argument_checks(lib, f32, status, kw):
    kw = dict(kw)
    if f32 and status == "FLA_ERR_ALIAS" and kw.get("ws") == DQ + TOK_B - 16:
        kw["ws"] = DQ + 2 * TOK_B - 16
    if f32 and status == "FLA_ERR_ALIAS" and kw.get("dq") == OUT + TOK_B - 16:
        kw["dq"] = OUT + 2 * TOK_B - 16
    assert _call_bwd(f32=f32, **kw) == _header_enum("FLA")[status]


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible (the calls would launch on fake pointers)")
def test_bwd_wide_windows_supported(lib):
    """Every argument check passes (the call gets as far as the device query) for windows of
    more than 256 tokens, also with RoPE: windows wider than the bf16 RoPE forward's 32 x 32
    cos / sin table take (cos, sin) per rotated piece."""
    codes = _header_enum("FLA")
    # 17 x 17 = 289 tokens per window: three 128-token blocks of the bf16 kernel; the fp32
    # kernels take it as well
    assert _call_bwd(window=17, shift=0) == codes["FLA_ERR_ARCH"]
    assert _call_bwd(f32=True, window=17, shift=0) == codes["FLA_ERR_ARCH"]
    for kw in (dict(window=17), dict(window=32), dict(window=33), dict(Hgrid=4, window=64),
               dict(Hgrid=64, Wgrid=64, window=64)):
        assert _call_rope_bwd(shift=0, **kw) == codes["FLA_ERR_ARCH"]
        assert fb.fla_swin_attn_rope_fwd(Q, K, V, OUT, 1, 12, kw.get("Hgrid", 64), kw.get("Wgrid", 64), 64,
                                         kw["window"], 0, 0, 1e4, 1.0, 0, check=False) == codes["FLA_ERR_ARCH"]


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible (the calls would launch on fake pointers)")
def test_bwd_mask_mode_needs_no_workspace(lib):
    codes = _header_enum("FLA")
    for kw in (dict(), dict(window=17, shift=0), dict(window=32, shift=16)):
        for f32 in (False, True):
            st = _call_bwd(f32=f32, ws=0, ws_bytes=0, **kw)
            assert st not in (codes["FLA_ERR_WORKSPACE"], codes["FLA_ERR_NULL"]), (kw, f32)
    assert _call_bwd(ws=0, ws_bytes=0, pad_mode=1) == codes["FLA_ERR_WORKSPACE"]


def test_bwd_workspace_size_examples(lib):
    # 64 x 64 grid, 12 heads, KV-token mode: window 16 shift 8 has 25 windows of up to 256
    # tokens (2 blocks of 128), window 32 shift 16 has 9 windows of up to 1024 (8 blocks), each
    # block with one 512-byte pad partial per head; MASK mode needs none
    assert fb.fla_swin_attn_bwd_workspace(1, 12, [(64, 64)], 16, 8, 1) == 25 * 2 * 12 * 512
    assert fb.fla_swin_attn_bwd_workspace(1, 12, [(64, 64)], 16, 8, 0) == 0
    assert fb.fla_swin_attn_bwd_workspace(1, 12, [(64, 64)], 32, 16, 0) == 0
    assert fb.fla_swin_attn_bwd_workspace(1, 12, [(64, 64)], 32, 16, 1) == 9 * 8 * 12 * 512


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
def test_training_entry_points_without_device_report_arch(lib):
    codes = _header_enum("FLA")
    assert _call_lse() == codes["FLA_ERR_ARCH"] and _call_lse(f32=True) == codes["FLA_ERR_ARCH"]
    assert _call_bwd() == codes["FLA_ERR_ARCH"] and _call_bwd(f32=True) == codes["FLA_ERR_ARCH"]
    assert _call_bwd(pad_mode=1) == codes["FLA_ERR_ARCH"]


def _call_noalloc(**kw):
    a = dict(GOOD)
    a.update({k: v for k, v in kw.items() if k in GOOD})
    p = dict(q=Q, k=K, v=V, out=OUT, dout=DOUT, lse=LSE, dq=DQ, dk=DK, dv=DV)
    p.update({k: v for k, v in kw.items() if k in p})
    return fb.fla_swin_attn_bwd_noalloc(p["q"], p["k"], p["v"], p["out"], p["dout"], p["lse"], p["dq"], p["dk"],
                                        p["dv"], a["B"], a["heads"], a["Hgrid"], a["Wgrid"], a["head_dim"],
                                        a["window"], a["shift"], a["pad_mode"], 0, check=False)


NOALLOC_CASES = [
    ("FLA_ERR_SHAPE", dict(B=-1)), ("FLA_ERR_NULL", dict(dout=0)), ("FLA_ERR_ALIGN", dict(dk=DK + 2)),
    ("FLA_ERR_HEAD_DIM", dict(head_dim=32)), ("FLA_ERR_SHIFT", dict(shift=16)),
    ("FLA_ERR_PAD_MODE", dict(pad_mode=2)), ("FLA_ERR_TOO_LARGE", dict(Hgrid=1 << 20, Wgrid=1 << 20)),
    # workspace beyond the static scratch: pad partials of 25 windows x 2 blocks x 12 heads
    # (300 KiB per batch entry: 40 entries fit, 160 do not), and of window-32 windows
    # (9 windows x 8 blocks x 12 heads, 432 KiB per entry)
    ("FLA_ERR_SCRATCH", dict(B=160, pad_mode=1)), ("FLA_ERR_SCRATCH", dict(B=64, window=32, shift=16, pad_mode=1)),
    ("FLA_ERR_ALIAS", dict(dq=Q)), ("FLA_ERR_ALIAS", dict(dv=DK + 64)),
]


@pytest.mark.parametrize("status,kw", NOALLOC_CASES, ids=["%s-%d" % (c[0], i) for i, c in enumerate(NOALLOC_CASES)])
def test_noalloc_argument_checks(lib, status, kw):
    """The allocation-free backward checks its arguments like the backward, and turns a
    workspace need beyond the static scratch into FLA_ERR_SCRATCH before touching a device."""
    assert _call_noalloc(**kw) == _header_enum("FLA")[status]


def test_noalloc_scratch_limit_matches_workspace_sizes(lib):
    """FLA_ERR_SCRATCH exactly when fla_swin_attn_bwd_workspace() exceeds FLA_SCRATCH_BYTES."""
    m = re.search(r"#define FLA_SCRATCH_BYTES \((\d+)u << (\d+)\)", open(HEADER).read())
    cap = int(m.group(1)) << int(m.group(2))
    assert cap == 16 << 20
    code = _header_enum("FLA")["FLA_ERR_SCRATCH"]
    for B, heads, window, shift, pm in ((1, 12, 16, 8, 1), (54, 12, 16, 8, 1), (55, 12, 16, 8, 1),
                                        (1, 12, 32, 16, 0), (37, 12, 32, 16, 1), (38, 12, 32, 16, 1)):
        need = fb.fla_swin_attn_bwd_workspace(B, heads, [(64, 64)], window, shift, pm)
        st = _call_noalloc(B=B, heads=heads, window=window, shift=shift, pad_mode=pm)
        assert (st == code) == (need > cap), (B, heads, window, need, st)


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
def test_noalloc_without_device_reports_arch(lib):
    codes = _header_enum("FLA")
    assert _call_noalloc() == codes["FLA_ERR_ARCH"] and _call_noalloc(pad_mode=1) == codes["FLA_ERR_ARCH"]
    assert _call_noalloc(heads=1, window=32, shift=16) == codes["FLA_ERR_ARCH"]


def test_empty_training_calls_are_ok(lib):
    assert _call_lse(B=0, lse=0, q=0) == 0
    assert _call_bwd(heads=0, dq=0, ws=0, ws_bytes=0) == 0
    assert _call_noalloc(B=0, dq=0) == 0


@pytest.mark.parametrize("grids,k,s,pm", [
    ([(256, 256)], 16, 8, 1), ([(64, 64)], 16, 8, 0), ([(150, 203)], 16, 8, 1),
    ([(128, 128), (32, 32)], 16, 8, 1), ([(40, 24)], 20, 10, 1), ([(3, 3)], 1, 0, 1)])
def test_bwd_workspace_size(lib, grids, k, s, pm):
    """KV-token mode: one pad-gradient partial (128 floats) per (batch entry, head, window,
    block of 128 tokens of the largest window); nothing in MASK mode."""
    B, heads = 2, 3
    n_win = sum(len(O.window_sizes(h, w, k, s)) for h, w in grids)
    nbb = max(-(-max(sz for h, w in grids for sz in O.window_sizes(h, w, k, s)) // 128), 1)
    want = B * heads * n_win * nbb * 128 * 4 if pm == 1 else 0
    assert fb.fla_swin_attn_bwd_workspace(B, heads, grids, k, s, pm) == want
    assert fb.fla_swin_attn_bwd_workspace(B, heads, grids, k, s, 0) == 0


def test_bwd_block_count_is_that_of_the_largest_window(lib):
    """The workspace counts blocks of the largest window exactly (first, last or a full window
    along each axis), for grids smaller and larger than the window and every shift."""
    rng = np.random.default_rng(5)
    for _ in range(300):
        k = int(rng.integers(1, 40))
        s = int(rng.integers(0, k))
        H, W = int(rng.integers(1, 90)), int(rng.integers(1, 90))
        sizes = O.window_sizes(H, W, k, s)
        want = len(sizes) * -(-max(sizes) // 128) * 128 * 4
        assert fb.fla_swin_attn_bwd_workspace(1, 1, [(H, W)], k, s, 1) == want, (H, W, k, s)


def test_bwd_workspace_errors(lib):
    codes = _header_enum("FLA")
    n = ctypes.c_size_t()
    arr = (ctypes.c_int * 2)(8, 8)
    assert lib.fla_swin_attn_bwd_workspace(1, 1, 1, arr, 4, 4, 1, ctypes.byref(n)) == codes["FLA_ERR_SHIFT"]
    assert lib.fla_swin_attn_bwd_workspace(1, 1, 1, arr, 4, 0, 1, None) == codes["FLA_ERR_NULL"]
    assert lib.fla_swin_attn_bwd_workspace(1, 1, 0, arr, 4, 0, 1, ctypes.byref(n)) == codes["FLA_ERR_SHAPE"]


@pytest.mark.parametrize("grids,k,s,pm", [
    ([(256, 256)], 16, 8, 0), ([(256, 256)], 16, 8, 1), ([(150, 203)], 16, 8, 0),
    ([(128, 128), (32, 32)], 16, 8, 1), ([(20, 13)], 8, 3, 1)])
def test_bwd_work_counts(lib, grids, k, s, pm):
    B, heads = 2, 12
    for eb in (2, 4):
        f, b = fb.fla_swin_attn_bwd_work(B, heads, grids, 64, k, s, pm, eb)
        f0, b0 = O.ms_work_counts(B, heads, grids, 64, k, s, pm, eb)
        L = sum(h * w for h, w in grids)
        assert f == 2.5 * f0                           # five products instead of two
        assert b == 2 * b0 + 4 * B * heads * L         # eight tensors instead of four, plus lse


# ---- RoPE forward ---------------------------------------------------------------------
def _call_rope(f32=False, theta=10000.0, scale=1.0, **kw):
    a = dict(GOOD)
    a.update({k: v for k, v in kw.items() if k in GOOD})
    p = dict(q=Q, k=K, v=V, out=OUT)
    p.update({k: v for k, v in kw.items() if k in p})
    return fb.fla_swin_attn_rope_fwd(p["q"], p["k"], p["v"], p["out"], a["B"], a["heads"], a["Hgrid"],
                                     a["Wgrid"], a["head_dim"], a["window"], a["shift"], a["pad_mode"],
                                     theta, scale, 0, check=False, f32=f32)


ROPE_CASES = [
    ("FLA_ERR_ROPE", dict(theta=0.0)), ("FLA_ERR_ROPE", dict(theta=-10.0)),
    ("FLA_ERR_ROPE", dict(theta=float("inf"))), ("FLA_ERR_ROPE", dict(theta=float("nan"))),
    ("FLA_ERR_ROPE", dict(scale=float("inf"))), ("FLA_ERR_ROPE", dict(scale=float("nan"))),
    ("FLA_ERR_PAD_MODE", dict(pad_mode=2, theta=0.0)),      # pad mode is checked first
    ("FLA_ERR_NULL", dict(q=0, theta=0.0)), ("FLA_ERR_ALIAS", dict(out=Q)),
]


@pytest.mark.parametrize("f32", [False, True], ids=["bf16", "f32"])
@pytest.mark.parametrize("status,kw", ROPE_CASES, ids=["%s-%d" % (c[0], i) for i, c in enumerate(ROPE_CASES)])
def test_rope_argument_checks(lib, f32, status, kw):
    assert _call_rope(f32=f32, **kw) == _header_enum("FLA")[status]


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
def test_rope_without_device_reports_arch(lib):
    codes = _header_enum("FLA")
    for kw in (dict(), dict(scale=0.0), dict(scale=-2.0, theta=1.0), dict(pad_mode=1)):
        assert _call_rope(**kw) == codes["FLA_ERR_ARCH"]
        assert _call_rope(f32=True, **kw) == codes["FLA_ERR_ARCH"]


# ---- tensor-level wrappers: shape checks before any device access -----------------------
class _FakeCuda:
    """Just enough of a tensor for the wrappers' checks (dtype, device flag, layout, shape)."""
    def __init__(self, shape, dtype=None):
        import torch
        self.shape = torch.Size(shape)
        self.dtype = dtype or torch.bfloat16
        self.is_cuda = True

    def is_contiguous(self):
        return True

    def dim(self):
        return len(self.shape)

    def reshape(self, *s):
        return _FakeCuda(s, self.dtype)


@pytest.mark.parametrize("qs,ks,pm", [
    ((1, 63, 2, 64), (1, 64, 2, 64), 0),       # q rows != H*W
    ((1, 64, 2, 64), (1, 64, 2, 64), 1),       # KV-token mode needs the pad row
    ((1, 64, 2, 64), (1, 65, 2, 64), 0),       # extra row without KV-token mode
    ((1, 64, 2, 64), (1, 64, 3, 64), 0),       # heads differ
    ((2, 64, 2, 64), (1, 64, 2, 64), 0),       # batch differs
])
def test_wrappers_reject_mismatched_shapes(qs, ks, pm):
    q, k = _FakeCuda(qs), _FakeCuda(ks)
    with pytest.raises(ValueError):
        fb.swin_attn(q, k, k, 8, 8, 4, 0, pm)
    with pytest.raises(ValueError):
        fb.swin_attn_ms(q, k, k, [(8, 8)], 4, 0, pm)
    with pytest.raises(ValueError):
        fb.swin_attn_fwd_train(q, k, k, [(8, 8)], 4, 0, pm)
    with pytest.raises(ValueError):
        fb.swin_attn_rope(q, k, k, 8, 8, 4, 0, pm)


def test_swin_attn_grid_of_a_5d_tensor_must_match():
    q = _FakeCuda((1, 8, 8, 2, 64))
    with pytest.raises(ValueError):
        fb.swin_attn(q, q, q, 8, 4, 4, 0)


def _call_rope_bwd(theta=10000.0, scale=1.0, **kw):
    a = dict(GOOD)
    a.update({k: v for k, v in kw.items() if k in GOOD})
    p = dict(q=Q, k=K, v=V, out=OUT, dout=DOUT, lse=LSE, dq=DQ, dk=DK, dv=DV, ws=WS)
    p.update({k: v for k, v in kw.items() if k in p})
    return fb.fla_swin_attn_rope_bwd(p["q"], p["k"], p["v"], p["out"], p["dout"], p["lse"], p["dq"], p["dk"],
                                     p["dv"], p["ws"], 1 << 24, a["B"], a["heads"], a["Hgrid"], a["Wgrid"],
                                     a["head_dim"], a["window"], a["shift"], a["pad_mode"], theta, scale, 0,
                                     check=False)


def test_rope_training_argument_checks(lib):
    codes = _header_enum("FLA")
    assert _call_rope_bwd(theta=0.0) == codes["FLA_ERR_ROPE"]
    assert _call_rope_bwd(scale=float("nan")) == codes["FLA_ERR_ROPE"]
    assert _call_rope_bwd(pad_mode=3, theta=0.0) == codes["FLA_ERR_PAD_MODE"]
    assert _call_rope_bwd(dq=Q) == codes["FLA_ERR_ALIAS"]
    assert fb.fla_swin_attn_rope_fwd_lse(Q, K, V, OUT, 0, 1, 12, 64, 64, 64, 16, 8, 0, 1e4, 1.0, 0,
                                         check=False) == codes["FLA_ERR_NULL"]
    assert fb.fla_swin_attn_rope_fwd_lse(Q, K, V, OUT, LSE, 1, 12, 64, 64, 64, 16, 8, 0, -1.0, 1.0, 0,
                                         check=False) == codes["FLA_ERR_ROPE"]
    if not _gpu_visible():
        assert _call_rope_bwd() == codes["FLA_ERR_ARCH"]
        assert fb.fla_swin_attn_rope_fwd_lse(Q, K, V, OUT, LSE, 1, 12, 64, 64, 64, 16, 8, 0, 1e4, 1.0, 0,
                                             check=False) == codes["FLA_ERR_ARCH"]


def test_rope_training_wrappers_check_before_launching():
    import torch
    q = _FakeCuda((1, 64, 2, 64), torch.float32)
    with pytest.raises(ValueError):   # RoPE training is bf16 only
        fb.swin_attn_rope_fwd_train(q, q, q, 8, 8, 4, 0)
    qb, kb = _FakeCuda((1, 63, 2, 64)), _FakeCuda((1, 64, 2, 64))
    with pytest.raises(ValueError):   # q rows != H*W
        fb.swin_attn_rope_fwd_train(qb, kb, kb, 8, 8, 4, 0)


def test_swin_attention_rope_takes_one_grid():
    q = _FakeCuda((1, 80, 2, 64))
    with pytest.raises(ValueError):
        fb.swin_attention(q, q, q, [(8, 8), (4, 4)], 4, 0, 0, rope=(1e4, 1.0))


# ---- Cycle-scan ------------------------------------------------------------------------------

_CS_BASE = 1 << 40   # fake device addresses, far apart (nothing is dereferenced)


def _cs_call(B=1, L=100, d=64, N=32, repeats=3, **over):
    nx, nb, na = B * L * d * 4, B * L * N * 4, d * N * 4
    p = {"x": _CS_BASE, "delta": _CS_BASE + (1 << 36), "A": _CS_BASE + (2 << 36), "Bm": _CS_BASE + (3 << 36),
         "Cm": _CS_BASE + (4 << 36), "y": _CS_BASE + (5 << 36), "ws": _CS_BASE + (6 << 36), "ws_bytes": 1 << 34}
    p.update(over)
    return fb.load_library().fla_cycle_scan(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["y"], p["ws"],
                                            p["ws_bytes"], B, L, d, N, repeats, None)


def _st(name):
    return _header_enum("FLA")[name]


@pytest.mark.parametrize("status,kw", [
    ("FLA_ERR_SHAPE", dict(B=-1)), ("FLA_ERR_SHAPE", dict(L=-1)), ("FLA_ERR_SHAPE", dict(d=-1)),
    ("FLA_ERR_SHAPE", dict(N=0)), ("FLA_ERR_SHAPE", dict(repeats=0)),
    ("FLA_ERR_NULL", dict(x=None)), ("FLA_ERR_NULL", dict(Cm=None)), ("FLA_ERR_NULL", dict(y=None)),
    ("FLA_ERR_ALIGN", dict(delta=_CS_BASE + (1 << 36) + 2)), ("FLA_ERR_ALIGN", dict(ws=_CS_BASE + (6 << 36) + 1)),
    ("FLA_ERR_UNSUPPORTED", dict(N=3)), ("FLA_ERR_UNSUPPORTED", dict(N=64)),
    ("FLA_ERR_TOO_LARGE", dict(B=1 << 10, L=1 << 20, d=1 << 10)),
    ("FLA_ERR_WORKSPACE", dict(ws=None)), ("FLA_ERR_WORKSPACE", dict(ws_bytes=16)),
    ("FLA_ERR_ALIAS", dict(y=_CS_BASE + 4)), ("FLA_ERR_ALIAS", dict(ws=_CS_BASE + (5 << 36) + 64)),
    ("FLA_ERR_ALIAS", dict(y=_CS_BASE + (2 << 36))),
])
def test_cycle_scan_argument_checks(lib, status, kw):
    assert _cs_call(**kw) == _st(status), kw


def test_cycle_scan_check_order(lib):
    # shape before null, null before alignment, alignment before the state count, ...
    assert _cs_call(N=0, x=None) == _st("FLA_ERR_SHAPE")
    assert _cs_call(x=None, delta=_CS_BASE + 2) == _st("FLA_ERR_NULL")
    assert _cs_call(N=3, delta=_CS_BASE + (1 << 36) + 2) == _st("FLA_ERR_ALIGN")
    assert _cs_call(N=3, ws=None) == _st("FLA_ERR_UNSUPPORTED")
    assert _cs_call(ws=None, y=_CS_BASE) == _st("FLA_ERR_WORKSPACE")


@pytest.mark.parametrize("kw", [dict(B=0), dict(L=0), dict(d=0)])
def test_cycle_scan_empty_is_ok_and_ignores_pointers(lib, kw):
    assert _cs_call(x=None, delta=None, A=None, Bm=None, Cm=None, y=None, ws=None, ws_bytes=0, **kw) == 0


def test_cycle_scan_inputs_may_alias(lib):
    # x, delta, Bm and Cm may share memory (they are only read); the outputs may not
    if not _gpu_visible():
        assert _cs_call(delta=_CS_BASE, Bm=_CS_BASE, Cm=_CS_BASE) == _st("FLA_ERR_ARCH")


@pytest.mark.skipif(_gpu_visible(), reason="a GPU is visible")
def test_cycle_scan_no_device_reports_arch(lib):
    assert _cs_call() == _st("FLA_ERR_ARCH")


@pytest.mark.parametrize("B,L,d,N", [(1, 65536, 768, 32), (2, 37, 70, 4), (1, 1, 1, 1), (3, 5000, 5, 16),
                                     (1, 2048, 64, 8), (1, 2049, 64, 8)])
def test_cycle_scan_workspace_size(lib, B, L, d, N):
    # chunks of T tokens, T the smallest power of two from 32 to 256 giving at most 64 chunks
    # (256 tokens past 16384); (N + 1) floats per (batch entry, chunk, channel)
    T = 32
    while T < 256 and T * 64 < L:
        T *= 2
    nch = -(-L // T)
    assert fb.fla_cycle_scan_workspace(B, L, d, N, 3) == 4 * B * nch * d * (N + 1)


def test_cycle_scan_workspace_errors(lib):
    n = ctypes.c_size_t()
    assert lib.fla_cycle_scan_workspace(1, 10, 4, 4, 3, None) == _st("FLA_ERR_NULL")
    assert lib.fla_cycle_scan_workspace(-1, 10, 4, 4, 3, ctypes.byref(n)) == _st("FLA_ERR_SHAPE")
    assert lib.fla_cycle_scan_workspace(1, 10, 4, 5, 3, ctypes.byref(n)) == _st("FLA_ERR_UNSUPPORTED")
    assert lib.fla_cycle_scan_workspace(0, 10, 4, 4, 3, ctypes.byref(n)) == 0 and n.value == 0


def test_cycle_scan_work_counts(lib):
    e, b = fb.fla_cycle_scan_work(2, 1000, 96, 16, 3)
    assert e == 2 * 1000 * 96 * 16
    assert b == 4 * (3 * 2 * 1000 * 96 + 2 * 2 * 1000 * 16 + 96 * 16)


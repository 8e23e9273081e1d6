"""Pins of the multi-scale oracle (HRSAM++, App. C): several token grids in one sequence,
each with its own shifted windows, and one pad token shared by all grids.

Each ``pin_ms_*`` takes the module ``oracle.multiscale`` so that the mutation test at the
end can hand in a patched copy; every planted mistake must fail at least one pin."""
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle as O
import oracle.multiscale as MS

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
PAD_MASK, PAD_KVTOKEN = O.PAD_MASK, O.PAD_KVTOKEN


def read_ms_golden():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "ms_index_mappings.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            key, *rest = line.split()
            if key == "case":
                kv = dict(t.split("=") for t in rest)
                grids = [tuple(map(int, g.split("x"))) for g in kv["grids"].split(",")]
                cur = {"grids": grids, "k": int(kv["k"]), "s": int(kv["s"])}
                cases.append(cur)
            else:
                cur[key] = [int(t) for t in rest]
    return cases


def _inputs(B, heads, grids, d, pad_mode, seed):
    rng = np.random.default_rng(seed)
    L = sum(h * w for h, w in grids)
    rows = L + (1 if pad_mode == PAD_KVTOKEN else 0)
    return (rng.standard_normal((B, L, heads, d)), rng.standard_normal((B, rows, heads, d)),
            rng.standard_normal((B, rows, heads, d)))


def _offsets(grids):
    """Row offsets computed here, not by the oracle."""
    offs, o = [], 0
    for h, w in grids:
        offs.append(o)
        o += h * w
    return offs, o


def _all_queries(B, grids):
    return np.array([(b, gi, y, x) for b in range(B) for gi, (h, w) in enumerate(grids)
                     for y in range(h) for x in range(w)])


def pin_ms_golden(M):
    for c in read_ms_golden():
        idx, lengths, inv = M.ms_shift_window_indices(c["grids"], c["k"], c["s"])
        kv, kvl = M.ms_kv_padding_indices(c["grids"], c["k"], c["s"])
        assert idx.tolist() == c["indices"]
        assert lengths.tolist() == c["lengths"]
        assert kv.tolist() == c["kv_indices"]
        assert kvl.tolist() == c["kv_lengths"]
        x = np.arange(len(idx)) * 5 + 1
        assert (x[idx][inv] == x).all()


def check_forms(M, grids, window, shift, pad_mode, seed=0):
    q, k, v = _inputs(2, 2, grids, 4, pad_mode, seed)
    a = M.swin_attention_ms(q, k, v, grids, window, shift, pad_mode)
    b = M.swin_attention_ms_fla(q, k, v, grids, window, shift, pad_mode)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    qs = _all_queries(2, grids)
    c = M.swin_attention_ms_at(q, k, v, grids, window, shift, pad_mode, qs)
    offs, _ = _offsets(grids)
    rows = np.array([offs[g] + y * grids[g][1] + x for _, g, y, x in qs])
    np.testing.assert_allclose(a[qs[:, 0], rows], c, rtol=0, atol=1e-12)


def pin_ms_forms(M):
    for grids, window, shift in [([(9, 7), (4, 5)], 4, 2), ([(6, 6), (3, 3), (2, 5)], 3, 1),
                                 ([(5, 8)], 4, 0), ([(8, 4), (8, 4)], 4, 3)]:
        for pad_mode in (PAD_MASK, PAD_KVTOKEN):
            check_forms(M, grids, window, shift, pad_mode)


def pin_ms_centroids(M):
    """q = k = 0: every real key of the window weighs the same, so out = mean of v over the
    query's region.  With v = (grid id, y, x), each output is the centroid of a region of
    its own grid."""
    grids = [(12, 10), (5, 7)]
    window, shift = 4, 2
    offs, L = _offsets(grids)
    q = np.zeros((1, L, 1, 3))
    k = np.zeros((1, L, 1, 3))
    v = np.zeros((1, L, 1, 3))
    for gi, (h, w) in enumerate(grids):
        yy, xx = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
        v[0, offs[gi]:offs[gi] + h * w, 0] = np.stack([np.full(h * w, gi), yy.ravel(), xx.ravel()], 1)
    out = M.swin_attention_ms(q, k, v, grids, window, shift, PAD_MASK)
    for gi, (h, w) in enumerate(grids):
        for y in range(h):
            for x in range(w):
                ry = [t for t in range(h) if (t - shift) // window == (y - shift) // window]
                rx = [t for t in range(w) if (t - shift) // window == (x - shift) // window]
                np.testing.assert_allclose(out[0, offs[gi] + y * w + x, 0], [gi, np.mean(ry), np.mean(rx)],
                                           atol=1e-12)


def pin_ms_shared_pad(M):
    """KV-token mode with q = k = 0: out = (sum of the region's v + n_pad * v_pad) / k^2, with
    one pad row (index L, after all grids) for every grid."""
    grids = [(6, 6), (3, 5)]
    window, shift = 4, 2
    offs, L = _offsets(grids)
    q = np.zeros((1, L, 1, 2))
    k = np.zeros((1, L + 1, 1, 2))
    v = np.random.default_rng(0).standard_normal((1, L + 1, 1, 2))
    out = M.swin_attention_ms(q, k, v, grids, window, shift, PAD_KVTOKEN)
    for gi, (h, w) in enumerate(grids):
        for y in range(h):
            for x in range(w):
                sel = [offs[gi] + yy * w + xx for yy in range(h) for xx in range(w)
                       if (yy - shift) // window == (y - shift) // window
                       and (xx - shift) // window == (x - shift) // window]
                want = (v[0, sel, 0].sum(0) + (window * window - len(sel)) * v[0, L, 0]) / window ** 2
                np.testing.assert_allclose(out[0, offs[gi] + y * w + x, 0], want, atol=1e-12)


def pin_ms_single_grid(M):
    for pad_mode in (PAD_MASK, PAD_KVTOKEN):
        q, k, v = _inputs(1, 3, [(20, 13)], 8, pad_mode, seed=3)
        a = M.swin_attention_ms(q, k, v, [(20, 13)], 8, 4, pad_mode)
        b = O.swin_attention_canvas(q, k, v, 20, 13, 8, 4, pad_mode)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


ALL_MS_PINS = [pin_ms_golden, pin_ms_forms, pin_ms_centroids, pin_ms_shared_pad, pin_ms_single_grid]


@pytest.mark.parametrize("pin", ALL_MS_PINS, ids=lambda p: p.__name__)
def test_ms_pin(pin):
    pin(MS)


grid_st = st.lists(st.tuples(st.integers(1, 13), st.integers(1, 13)), min_size=1, max_size=3)


@settings(max_examples=40, deadline=None)
@given(grids=grid_st, window=st.integers(1, 9), data=st.data(), pad_mode=st.sampled_from([0, 1]))
def test_ms_forms_agree_random(grids, window, data, pad_mode):
    shift = data.draw(st.integers(0, window - 1))
    check_forms(MS, grids, window, shift, pad_mode, seed=len(grids) * 100 + window)


def test_ms_work_counts():
    grids = [(64, 64), (32, 32)]
    f, b = O.ms_work_counts(1, 12, grids, 64, 16, 8, 0, 2)
    f0, b0 = O.work_counts(1, 12, 64, 64, 64, 16, 8, 0, 2)
    f1, b1 = O.work_counts(1, 12, 32, 32, 64, 16, 8, 0, 2)
    assert f == f0 + f1 and b == b0 + b1
    _, bk = O.ms_work_counts(1, 12, grids, 64, 16, 8, 1, 2)
    assert bk == b + 2 * 12 * 64 * 2     # one shared pad row of k and v, not one per grid


# ---- planted mistakes ----------------------------------------------------------------
_orig_sw = MS.ms_shift_window_indices
_orig_kv = MS.ms_kv_padding_indices


def _sw_no_offset(grids, k, s):
    idx, lens = [], []
    for h, w in grids:
        i, l, _ = MS.fla_shift_window_indices(h, w, k, s)
        idx.append(i)
        lens.append(l)
    i = np.concatenate(idx)
    return i, np.concatenate(lens), np.argsort(i, kind="stable")


def _kv_pad_per_grid(grids, k, s):
    offs, L = MS.grid_offsets(grids)
    idx, lens = [], []
    for (h, w), o in zip(grids, offs):
        i, l = MS.fla_kv_padding_indices(h, w, k, s)
        idx.append(np.minimum(i + o, L))
        lens.append(l)
    return np.concatenate(idx), np.concatenate(lens)


def _ms_pad_row_per_grid(q, k, v, grids, window, shift, pad_mode=PAD_MASK):
    offs, L = MS.grid_offsets(grids)
    out = np.empty_like(np.asarray(q, dtype=np.float64))
    for (h, w), o in zip(grids, offs):
        rows = slice(o, o + h * w)
        pr = min(o + h * w, L)
        kg = np.concatenate([k[:, rows], k[:, pr:pr + 1]], axis=1) if pad_mode else k[:, rows]
        vg = np.concatenate([v[:, rows], v[:, pr:pr + 1]], axis=1) if pad_mode else v[:, rows]
        out[:, rows] = MS.swin_attention_textbook(q[:, rows], kg, vg, h, w, window, shift, pad_mode)
    return out


def _offsets_reversed(grids):
    g = list(grids)[::-1]
    offs = np.concatenate([[0], np.cumsum([h * w for h, w in g])]).astype(np.int64)
    return offs[:-1][::-1].copy(), int(offs[-1])


MS_MUTANTS = {
    "index_offset_missing": {"ms_shift_window_indices": _sw_no_offset},
    "pad_row_per_grid_in_index_list": {"ms_kv_padding_indices": _kv_pad_per_grid},
    "pad_row_per_grid_in_composition": {"swin_attention_ms": _ms_pad_row_per_grid},
    "grid_offsets_reversed": {"grid_offsets": _offsets_reversed},
    "region_ignores_shift": {"_region": lambda c, k, s: np.floor_divide(np.asarray(c), k)},
}


@pytest.mark.parametrize("name", sorted(MS_MUTANTS))
def test_ms_pins_catch_mutant(name, monkeypatch):
    for attr, repl in MS_MUTANTS[name].items():
        monkeypatch.setattr(MS, attr, repl)
    failed = []
    for pin in ALL_MS_PINS:
        try:
            pin(MS)
        except Exception as e:
            failed.append((pin.__name__, type(e).__name__))
    assert failed, "mutant %s passed every multi-scale pin" % name

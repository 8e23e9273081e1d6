"""CPU tests of the fp64 oracle against its pins (see oracle_pins) and across its forms."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle as O
import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(O)


def test_centroids_all_forms():
    P.pin_centroids(O, forms=("swin_attention_textbook", "swin_attention_canvas",
                              "swin_attention_fla", "swin_attention_bruteforce"))


@pytest.mark.parametrize("form", ["swin_attention_canvas", "swin_attention_fla",
                                  "swin_attention_bruteforce"])
def test_closed_forms_other_forms(form):
    P.pin_global(O, form)
    P.pin_wmsa(O, form)
    P.pin_constant_v(O, form)
    P.pin_roll_invariant(O, form)
    P.pin_kvtoken_zero_canvas(O, form)


@st.composite
def _case(draw):
    k = draw(st.integers(1, 9))
    s = draw(st.integers(0, k - 1))
    H = draw(st.integers(1, 14))
    W = draw(st.integers(1, 14))
    return (draw(st.integers(1, 2)), draw(st.integers(1, 2)), H, W, draw(st.integers(1, 6)), k, s,
            draw(st.sampled_from([O.PAD_MASK, O.PAD_KVTOKEN])), draw(st.integers(0, 2**31 - 1)))


@settings(max_examples=80, deadline=None)
@given(_case())
def test_forms_agree(case):
    B, heads, H, W, d, k, s, pad_mode, seed = case
    rng = np.random.default_rng(seed)
    extra = 1 if pad_mode == O.PAD_KVTOKEN else 0
    q = rng.standard_normal((B, H * W, heads, d))
    kk = rng.standard_normal((B, H * W + extra, heads, d))
    v = rng.standard_normal((B, H * W + extra, heads, d))
    ref = O.swin_attention_bruteforce(q, kk, v, H, W, k, s, pad_mode)
    assert np.isfinite(ref).all()
    for fn in (O.swin_attention_textbook, O.swin_attention_canvas, O.swin_attention_fla):
        np.testing.assert_allclose(fn(q, kk, v, H, W, k, s, pad_mode), ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("H,W,k,s", [(64, 64, 16, 8), (150, 203, 16, 8), (32, 32, 8, 4),
                                     (32, 32, 8, 0), (13, 1, 4, 3), (1, 1, 16, 8), (33, 17, 5, 2)])
def test_index_properties(H, W, k, s):
    """App. A: the Q mapping is a bijection with inverse argsort; lengths add up to L.
    App. B: every KV segment has k*k entries, virtual slots point at row L."""
    idx, lengths, inv = O.fla_shift_window_indices(H, W, k, s)
    L = H * W
    assert sorted(idx.tolist()) == list(range(L))
    x = np.arange(L) * 3 + 1
    assert (x[idx][inv] == x).all()
    assert lengths.sum() == L and (lengths >= 1).all() and (lengths <= k * k).all()
    kv, kvl = O.fla_kv_padding_indices(H, W, k, s)
    assert (kvl == k * k).all() and len(kv) == kvl.sum()
    assert ((kv >= 0) & (kv <= L)).all()
    real = kv[kv < L]
    assert (real == idx).all()          # real KV slots come in the Q order
    assert (kv == L).sum() == len(kv) - L


def test_region_rule_matches_shifted_canvas():
    """Sec. 3.3: the canvas with k - s virtual tokens in front gives region floor((c-s)/k)."""
    for H, k, s in [(64, 16, 8), (20, 8, 3), (7, 4, 0), (5, 8, 7)]:
        idx, lengths, _ = O.fla_shift_window_indices(H, 1, k, s)
        seg = np.repeat(np.arange(len(lengths)), lengths)
        region = np.empty(H, dtype=np.int64)
        region[idx] = seg
        want = np.floor_divide(np.arange(H) - s, k)
        # same partition: region ids are an increasing relabelling of want
        assert (np.diff(region) >= 0).all()
        assert ((np.diff(region) > 0) == (np.diff(want) > 0)).all()


def test_work_counts_kvtoken():
    f0, b0 = O.work_counts(1, 12, 64, 64, 64, 16, 8, O.PAD_MASK, 2)
    f1, b1 = O.work_counts(1, 12, 64, 64, 64, 16, 8, O.PAD_KVTOKEN, 2)
    # 16 non-full windows (4 x 64 + 12 x 128 tokens = 1792 queries) gain one pad key each
    assert f1 - f0 == 4 * 64 * 12 * 1792
    assert b0 == 4 * 4096 * 12 * 64 * 2 and b1 - b0 == 2 * 12 * 64 * 2


def test_sampled_form_matches_full():
    rng = np.random.default_rng(3)
    H, W, k, s = 20, 13, 8, 4
    for pad_mode in (O.PAD_MASK, O.PAD_KVTOKEN):
        extra = 1 if pad_mode else 0
        q = rng.standard_normal((2, H * W, 3, 8))
        kk = rng.standard_normal((2, H * W + extra, 3, 8))
        v = rng.standard_normal((2, H * W + extra, 3, 8))
        full = O.swin_attention_textbook(q, kk, v, H, W, k, s, pad_mode)
        pts = np.array([[0, 0, 0], [1, 19, 12], [1, 3, 4], [0, 11, 7]])
        got = O.swin_attention_at(q, kk, v, H, W, k, s, pad_mode, pts)
        for n, (b, y, x) in enumerate(pts):
            np.testing.assert_allclose(got[n], full[b, y * W + x], rtol=0, atol=1e-12)

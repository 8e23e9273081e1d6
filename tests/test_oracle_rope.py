"""Pins of the fp64 RoPE oracle (``oracle.rope``) and planted mistakes they must catch (CPU).

Pins: hand-derived rotations (tests/golden/rope_small.txt); the same rotation written as a
complex multiplication of channel pairs with positions and frequencies computed here; norm
preservation per channel pair; scale 0 reduces to the plain textbook attention; and the
property RoPE exists for -- attention logits depend only on relative positions, so shifting
every coordinate by a constant leaves the MASK-mode output unchanged.  The sampled-query form
and the log-sum-exp are pinned against the whole-grid form and against facts computed here from
this file's own complex-form rotation: the one-hot readout (values e_j make out[i, j] the
attention probability, so LSE_i = z_ij + log w_j - log P_ij) and, in the global case, scipy's
logsumexp (Sec. 3.1 RoPE; Eq. 1)."""
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle.rope as R
from oracle import swin_oracle as SO

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "rope_small.txt")


def _golden_rows():
    env = {"cos": math.cos, "sin": math.sin}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, vin, vout = (p.split() for p in line.split("|"))
        H, W = int(head[0]), int(head[1])
        theta, scale = float(head[2]), float(head[3])
        tok, y, x = int(head[4]), int(head[5]), int(head[6])
        yield H, W, theta, scale, tok, y, x, [float(t) for t in vin], [eval(t, env) for t in vout]


def pin_golden(M):
    for H, W, theta, scale, tok, y, x, vin, vout in _golden_rows():
        assert tok == y * W + x
        xs = np.zeros((1, H * W, 1, 8))
        xs[0, tok, 0] = vin
        got = M.apply_rope(xs, H, W, theta, scale)[0, tok, 0]
        np.testing.assert_allclose(got, vout, rtol=0, atol=1e-14)


def pin_complex_form(M):
    rng = np.random.default_rng(31)
    for H, W, d, theta, scale in ((5, 7, 16, 10000.0, 1.0), (4, 3, 64, 500.0, 0.25), (2, 9, 8, 10.0, 3.0)):
        x = rng.standard_normal((2, H * W, 3, d))
        got = M.apply_rope(x, H, W, theta, scale)
        half = d // 2
        freqs = np.array([theta ** (-(2.0 * j) / half) for j in range(half // 2)])
        for t in range(H * W):
            y, xx = divmod(t, W)
            ang = np.concatenate([scale * y * freqs, scale * xx * freqs])
            z = x[:, t, :, 0::2] + 1j * x[:, t, :, 1::2]
            zr = z * np.exp(1j * ang)
            np.testing.assert_allclose(got[:, t, :, 0::2], zr.real, atol=1e-12)
            np.testing.assert_allclose(got[:, t, :, 1::2], zr.imag, atol=1e-12)


def pin_norms_and_pad_row(M):
    rng = np.random.default_rng(32)
    x = rng.standard_normal((1, 6 * 5 + 1, 2, 16))
    got = M.apply_rope(x, 6, 5, 10000.0, 1.0)
    n_in = x[:, :30, :, 0::2] ** 2 + x[:, :30, :, 1::2] ** 2
    n_out = got[:, :30, :, 0::2] ** 2 + got[:, :30, :, 1::2] ** 2
    np.testing.assert_allclose(n_out, n_in, rtol=1e-12)
    np.testing.assert_array_equal(got[:, 30], x[:, 30])      # the pad token has no position


def pin_scale_zero_is_plain(M):
    rng = np.random.default_rng(33)
    for pm in (0, 1):
        q = rng.standard_normal((1, 42, 2, 16))
        k = rng.standard_normal((1, 42 + pm, 2, 16))
        v = rng.standard_normal((1, 42 + pm, 2, 16))
        np.testing.assert_allclose(M.swin_attention_rope(q, k, v, 6, 7, 4, 2, pm, 10000.0, 0.0),
                                   SO.swin_attention_textbook(q, k, v, 6, 7, 4, 2, pm), atol=1e-13)


def pin_relative_positions(M):
    rng = np.random.default_rng(34)
    for H, W, k, s, d in ((9, 7, 4, 2, 16), (8, 8, 8, 4, 64)):
        q = rng.standard_normal((1, H * W, 2, d))
        kk = rng.standard_normal((1, H * W, 2, d))
        v = rng.standard_normal((1, H * W, 2, d))
        base = M.swin_attention_rope(q, kk, v, H, W, k, s, 0, 100.0, 1.0)
        moved = M.swin_attention_rope(q, kk, v, H, W, k, s, 0, 100.0, 1.0, y0=5.0, x0=-3.0)
        np.testing.assert_allclose(moved, base, atol=1e-12)
        # and RoPE does change the result (the pin is not vacuous)
        assert np.abs(base - SO.swin_attention_textbook(q, kk, v, H, W, k, s, 0)).max() > 1e-3


def pin_inverse(M):
    rng = np.random.default_rng(35)
    x = rng.standard_normal((2, 6 * 7 + 1, 3, 16))
    back = M.apply_rope(M.apply_rope(x, 6, 7, 100.0, 0.7), 6, 7, 100.0, 0.7, inverse=True)
    np.testing.assert_allclose(back, x, atol=1e-12)


def pin_rope_bwd_fd(M):
    """Gradients of the RoPE attention against central finite differences of its forward."""
    rng = np.random.default_rng(36)
    for H, W, k, s, pm in ((6, 5, 4, 2, 0), (6, 5, 4, 2, 1), (5, 7, 8, 3, 1)):
        L = H * W
        q = rng.standard_normal((1, L, 2, 8))
        kk = rng.standard_normal((1, L + pm, 2, 8))
        v = rng.standard_normal((1, L + pm, 2, 8))
        do = rng.standard_normal((1, L, 2, 8))
        dq, dk, dv = M.swin_attention_rope_bwd(q, kk, v, do, H, W, k, s, pm, 50.0, 0.8)
        U = [rng.standard_normal(t.shape) for t in (q, kk, v)]
        f = lambda t: float((do * M.swin_attention_rope(q + t * U[0], kk + t * U[1], v + t * U[2], H, W, k, s, pm,
                                                        50.0, 0.8)).sum())
        h = 1e-5
        fd = (f(h) - f(-h)) / (2 * h)
        an = float((dq * U[0]).sum() + (dk * U[1]).sum() + (dv * U[2]).sum())
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), ((H, W, k, s, pm), fd, an)
        lse = M.swin_attention_rope_lse(q, kk, v, H, W, k, s, pm, 50.0, 0.8)
        assert lse.shape == (1, 2, L) and np.isfinite(lse).all()


def _rotate_here(x, H, W, theta, scale):
    """RoPE written independently of the oracle: each adjacent channel pair of the first (second)
    half of a head is a complex number turned by scale * row (column) * theta^(-2j / (d/2));
    rows past H * W (the pad token) stay as they are."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    freqs = np.array([theta ** (-(2.0 * j) / half) for j in range(half // 2)])
    out = x.copy()
    for t in range(H * W):
        y, xx = divmod(t, W)
        ang = np.concatenate([scale * y * freqs, scale * xx * freqs])
        z = (x[:, t, :, 0::2] + 1j * x[:, t, :, 1::2]) * np.exp(1j * ang)
        out[:, t, :, 0::2], out[:, t, :, 1::2] = z.real, z.imag
    return out


def pin_rope_at_matches_full(M):
    """The sampled-query form equals the whole-grid form at every sampled query, both pad modes,
    with a base and scale other than the defaults (so both must be passed through)."""
    rng = np.random.default_rng(37)
    for H, W, k, s, pm in ((9, 7, 4, 2, 0), (9, 7, 4, 2, 1), (6, 10, 8, 3, 1), (5, 5, 8, 0, 0)):
        L = H * W
        q = rng.standard_normal((2, L, 2, 16))
        kk = rng.standard_normal((2, L + pm, 2, 16))
        v = rng.standard_normal((2, L + pm, 2, 16))
        full = M.swin_attention_rope(q, kk, v, H, W, k, s, pm, 40.0, 0.6)
        qs = np.array([(b, y, x) for b in range(2) for y in range(H) for x in range(W)
                       if (b * 7 + y * 3 + x) % 4 == 0])
        got = M.swin_attention_rope_at(q, kk, v, H, W, k, s, pm, qs, 40.0, 0.6)
        want = full[qs[:, 0], qs[:, 1] * W + qs[:, 2]]
        np.testing.assert_allclose(got, want, atol=1e-12, err_msg=str((H, W, k, s, pm)))


def pin_rope_lse_one_hot(M):
    """LSE of the RoPE attention read off the textbook attention of inputs rotated by this file's
    own rotation with one-hot values (out[i, j] = P_ij); a second, global case against scipy."""
    rng = np.random.default_rng(38)
    theta, scale = 30.0, 0.7
    for H, W, k, s, pm in ((5, 7, 4, 2, 0), (5, 7, 4, 2, 1), (7, 5, 8, 3, 1)):
        L = H * W
        d = 36                                   # >= L + 1 keys, a multiple of 4
        q = rng.standard_normal((1, L, 1, d))
        kk = rng.standard_normal((1, L + pm, 1, d))
        v = np.zeros_like(kk)
        v[0, np.arange(L + pm), 0, np.arange(L + pm)] = 1.0
        qr, kr = _rotate_here(q, H, W, theta, scale), _rotate_here(kk, H, W, theta, scale)
        out = SO.swin_attention_textbook(qr, kr, v, H, W, k, s, pm)       # out[0, i, 0, j] = P_ij
        lse = M.swin_attention_rope_lse(q, kk, v, H, W, k, s, pm, theta, scale)
        c = 1.0 / math.sqrt(d)
        for i in range(L):
            j = int(np.argmax(out[0, i, 0]))
            w = 1.0
            if j == L:
                w = float(k * k - np.count_nonzero(out[0, i, 0, :L] > 0))
            want = c * float(qr[0, i, 0] @ kr[0, j, 0]) + math.log(w) - math.log(out[0, i, 0, j])
            assert abs(lse[0, 0, i] - want) < 1e-10, ((H, W, k, s, pm), i, lse[0, 0, i], want)
    H, W, d = 4, 6, 8
    q = rng.standard_normal((2, H * W, 3, d))
    kk = rng.standard_normal((2, H * W, 3, d))
    v = rng.standard_normal((2, H * W, 3, d))
    lse = M.swin_attention_rope_lse(q, kk, v, H, W, 7, 0, 0, theta, scale)
    qr, kr = _rotate_here(q, H, W, theta, scale), _rotate_here(kk, H, W, theta, scale)
    z = np.einsum("bihd,bjhd->bhij", qr, kr) / math.sqrt(d)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=-1), rtol=1e-12, atol=1e-12)


PINS = [pin_golden, pin_complex_form, pin_norms_and_pad_row, pin_scale_zero_is_plain, pin_relative_positions,
        pin_inverse, pin_rope_bwd_fd, pin_rope_at_matches_full, pin_rope_lse_one_hot]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(R)


_orig_angles = R.rope_angles


def _angles_axes_swapped(H, W, d, theta=10000.0, scale=1.0, y0=0.0, x0=0.0):
    a = _orig_angles(H, W, d, theta, scale, y0, x0)
    q = a.shape[1] // 2
    return np.concatenate([a[:, q:], a[:, :q]], axis=1)


def _angles_sign(H, W, d, theta=10000.0, scale=1.0, y0=0.0, x0=0.0):
    return -_orig_angles(H, W, d, theta, scale, y0, x0)


def _angles_freq_over_d(H, W, d, theta=10000.0, scale=1.0, y0=0.0, x0=0.0):
    # frequency exponent 2j/d instead of 2j/(d/2)
    freq = float(theta) ** (-2.0 * np.arange(d // 4) / d)
    ys = (np.arange(H) + y0) * scale
    xs = (np.arange(W) + x0) * scale
    return np.concatenate([np.repeat(ys, W)[:, None] * freq, np.tile(xs, H)[:, None] * freq], axis=1)


def _angles_no_scale(H, W, d, theta=10000.0, scale=1.0, y0=0.0, x0=0.0):
    return _orig_angles(H, W, d, theta, 1.0, y0, x0)


def _apply_half_split(x, H, W, theta=10000.0, scale=1.0, y0=0.0, x0=0.0, inverse=False):
    # pairs (j, j + d/4) within each half instead of adjacent channels
    x = np.asarray(x, dtype=np.float64)
    B, rows, heads, d = x.shape
    perm = np.concatenate([np.stack([np.arange(h0, h0 + d // 4), np.arange(h0 + d // 4, h0 + d // 2)], 1).ravel()
                           for h0 in (0, d // 2)])
    inv = np.argsort(perm)
    return _orig_apply(x[..., perm], H, W, theta, scale, y0, x0, inverse)[..., inv]


def _apply_rotates_pad(x, H, W, theta=10000.0, scale=1.0, y0=0.0, x0=0.0, inverse=False):
    x = np.asarray(x, dtype=np.float64)
    out = _orig_apply(x, H, W, theta, scale, y0, x0, inverse)
    if x.shape[1] > H * W:   # rotate the pad row as if it were the token after the grid
        ext = np.zeros((x.shape[0], (H + 1) * W) + x.shape[2:])
        ext[:, :H * W + 1] = x[:, :H * W + 1]
        out[:, H * W] = _orig_apply(ext, H + 1, W, theta, scale, y0, x0, inverse)[:, H * W]
    return out


_orig_apply = R.apply_rope

def _apply_no_inverse(x, H, W, theta=10000.0, scale=1.0, y0=0.0, x0=0.0, inverse=False):
    return _orig_apply(x, H, W, theta, scale, y0, x0)


def _apply_inverse_skipped_on_pad(x, H, W, theta=10000.0, scale=1.0, y0=0.0, x0=0.0, inverse=False):
    out = _orig_apply(x, H, W, theta, scale, y0, x0, inverse)
    if inverse and out.shape[1] > H * W:
        out[:, H * W] = 0.0      # drops the pad token's gradient on the way back
    return out


_orig_at = R.swin_attention_rope_at
_orig_lse = R.swin_attention_rope_lse


def _at_k_unrotated(q, k, v, H, W, window, shift, pad_mode, queries, theta=10000.0, scale=1.0):
    return SO.swin_attention_at(_orig_apply(q, H, W, theta, scale), k, v, H, W, window, shift, pad_mode, queries)


def _at_scale_dropped(q, k, v, H, W, window, shift, pad_mode, queries, theta=10000.0, scale=1.0):
    return _orig_at(q, k, v, H, W, window, shift, pad_mode, queries, theta, 1.0)


def _at_theta_dropped(q, k, v, H, W, window, shift, pad_mode, queries, theta=10000.0, scale=1.0):
    return _orig_at(q, k, v, H, W, window, shift, pad_mode, queries, 10000.0, scale)


def _lse_k_unrotated(q, k, v, H, W, window, shift, pad_mode=0, theta=10000.0, scale=1.0):
    from oracle.backward import swin_attention_lse
    return swin_attention_lse(_orig_apply(q, H, W, theta, scale), k, v, H, W, window, shift, pad_mode)


def _lse_scale_dropped(q, k, v, H, W, window, shift, pad_mode=0, theta=10000.0, scale=1.0):
    return _orig_lse(q, k, v, H, W, window, shift, pad_mode, theta, 1.0)


def _lse_theta_dropped(q, k, v, H, W, window, shift, pad_mode=0, theta=10000.0, scale=1.0):
    return _orig_lse(q, k, v, H, W, window, shift, pad_mode, 10000.0, scale)


MUTANTS = {
    "at_k_unrotated": {"swin_attention_rope_at": _at_k_unrotated},
    "at_scale_dropped": {"swin_attention_rope_at": _at_scale_dropped},
    "at_theta_dropped": {"swin_attention_rope_at": _at_theta_dropped},
    "lse_k_unrotated": {"swin_attention_rope_lse": _lse_k_unrotated},
    "lse_scale_dropped": {"swin_attention_rope_lse": _lse_scale_dropped},
    "lse_theta_dropped": {"swin_attention_rope_lse": _lse_theta_dropped},
    "inverse_is_forward": {"apply_rope": _apply_no_inverse},
    "pad_gradient_dropped": {"apply_rope": _apply_inverse_skipped_on_pad},
    "axes_swapped": {"rope_angles": _angles_axes_swapped},
    "rotation_sign": {"rope_angles": _angles_sign},
    "frequency_exponent_over_d": {"rope_angles": _angles_freq_over_d},
    "scale_ignored": {"rope_angles": _angles_no_scale},
    "pairs_half_split": {"apply_rope": _apply_half_split},
    "pad_row_rotated": {"apply_rope": _apply_rotates_pad},
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    for attr, fn in MUTANTS[name].items():
        monkeypatch.setattr(R, attr, fn)
    failed = []
    for pin in PINS:
        try:
            pin(R)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, "mutant %s passed every pin" % name

"""Pins of the fp64 Cycle-scan oracle (``oracle.cycle_scan``) and planted mistakes they must catch (CPU).

Pins: hand-derived scans (tests/golden/cycle_scan_small.txt); the zero-order hold against the
matrix exponential of the augmented system [[a, b], [0, 0]] (van Loan), which gives the exact
one-step solution of h' = a h + b x for a held input, a = 0 included; the whole scan written
as a lower-triangular matrix, M[t, s] = sum_n C_t[n] exp(a[n] (cum_t - cum_s)) Bbar_s[n] with
cum the running sum of Delta, so that the products of Abar are never formed step by step;
the same matrix over the repeated sequence for Cycle-scan; and properties: one copy is the
plain scan, the output is linear in x, and with no memory (Abar = 0) every token gives
`repeats` times C . Bbar x (Sec. 3.5, the SSM equations and the Cycle-scan strategy)."""
import math
import os

import numpy as np
import pytest
import scipy.linalg

import oracle.cycle_scan as C

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "cycle_scan_small.txt")


def _golden_cases():
    env = {"log": math.log}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, a, delta, b, c, x, y = [f.split() for f in line.split("|")]
        L, d, N, r = map(int, head)
        ev = lambda fs: np.array([eval(f, env) for f in fs], dtype=np.float64)
        yield (L, d, N, r, ev(a).reshape(d, N), ev(delta).reshape(1, L, d), ev(b).reshape(1, L, N),
               ev(c).reshape(1, L, N), ev(x).reshape(1, L, d), ev(y).reshape(1, L, d))


def _inputs(rng, nb, L, d, N):
    x = rng.standard_normal((nb, L, d))
    delta = np.log1p(np.exp(rng.standard_normal((nb, L, d)) - 1.0))      # softplus: positive steps
    A = -rng.uniform(0.2, 3.0, (d, N))
    Bm = rng.standard_normal((nb, L, N))
    Cm = rng.standard_normal((nb, L, N))
    return x, delta, A, Bm, Cm


def _matrix_form(x, delta, A, Bm, Cm):
    """y from the explicit lower-triangular operator of the scan (no step recurrence)."""
    nb, L, d = x.shape
    y = np.zeros((nb, L, d))
    cum = np.cumsum(delta, axis=1)                                         # [nb, L, d]
    for bi in range(nb):
        for ch in range(d):
            a = A[ch]                                                      # [N]
            dl = delta[bi, :, ch]
            bbar = (np.exp(dl[:, None] * a[None, :]) - 1.0) / a[None, :] * Bm[bi]   # [L, N]
            gap = cum[bi, :, ch][:, None] - cum[bi, :, ch][None, :]        # [t, s]
            decay = np.exp(gap[:, :, None] * a[None, None, :])             # [t, s, N]
            Mts = np.einsum("tn,tsn,sn->ts", Cm[bi], decay, bbar) * np.tril(np.ones((L, L)))
            y[bi, :, ch] = Mts @ x[bi, :, ch]
    return y


def pin_golden(M):
    for L, d, N, r, a, delta, b, c, x, y in _golden_cases():
        got = M.cycle_scan(x, delta, a, b, c, r)
        np.testing.assert_allclose(got, y, rtol=1e-12, atol=1e-12, err_msg="golden %s" % ((L, d, N, r),))
        if r == 1:
            np.testing.assert_allclose(M.selective_scan(x, delta, a, b, c)[0], y, rtol=1e-12, atol=1e-12)


def pin_zoh_van_loan(M):
    rng = np.random.default_rng(11)
    for a, dl, b in [(-1.3, 0.7, 2.0), (0.0, 0.25, -3.0), (-25.0, 0.01, 1.5), (0.4, 1.1, 0.5)] + \
            [tuple(v) for v in zip(-rng.uniform(0, 5, 6), rng.uniform(0.01, 2, 6), rng.standard_normal(6))]:
        e = scipy.linalg.expm(np.array([[a * dl, b * dl], [0.0, 0.0]]))
        abar, bbar = M.zoh(np.array(dl), np.array([a]), np.array([b]))
        assert abs(abar[0] - e[0, 0]) < 1e-12 * max(1, abs(e[0, 0])), (a, dl, b)
        assert abs(bbar[0] - e[0, 1]) < 1e-12 * max(1, abs(e[0, 1])), (a, dl, b, bbar, e)


def pin_scan_matrix_form(M):
    rng = np.random.default_rng(12)
    x, delta, A, Bm, Cm = _inputs(rng, 2, 9, 3, 4)
    y, h = M.selective_scan(x, delta, A, Bm, Cm)
    np.testing.assert_allclose(y, _matrix_form(x, delta, A, Bm, Cm), rtol=1e-10, atol=1e-10)


def pin_cycle_matrix_form(M):
    rng = np.random.default_rng(13)
    x, delta, A, Bm, Cm = _inputs(rng, 2, 7, 3, 5)
    L = x.shape[1]
    for r in (1, 2, 3, 4):
        t = lambda v: np.concatenate([v] * r, axis=1)
        yl = _matrix_form(t(x), t(delta), A, t(Bm), t(Cm))
        want = yl.reshape(2, r, L, 3).sum(axis=1)
        np.testing.assert_allclose(M.cycle_scan(x, delta, A, Bm, Cm, r), want, rtol=1e-10, atol=1e-10,
                                   err_msg="repeats %d" % r)


def pin_cycle_properties(M):
    rng = np.random.default_rng(14)
    x, delta, A, Bm, Cm = _inputs(rng, 1, 11, 4, 3)
    np.testing.assert_allclose(M.cycle_scan(x, delta, A, Bm, Cm, 1), M.selective_scan(x, delta, A, Bm, Cm)[0],
                               rtol=1e-13, atol=1e-13)
    x2 = rng.standard_normal(x.shape)
    lhs = M.cycle_scan(2.0 * x - 3.0 * x2, delta, A, Bm, Cm, 3)
    rhs = 2.0 * M.cycle_scan(x, delta, A, Bm, Cm, 3) - 3.0 * M.cycle_scan(x2, delta, A, Bm, Cm, 3)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-10, atol=1e-10)
    # no memory: Abar = exp(-200) ~ 0, so every token contributes alone, `repeats` times
    Afast = np.full_like(A, -200.0)
    d1 = np.ones_like(delta)
    bbar_c = np.einsum("bln,bln->bl", (np.expm1(-200.0) / -200.0) * Bm, Cm)
    np.testing.assert_allclose(M.cycle_scan(x, d1, Afast, Bm, Cm, 3), 3.0 * bbar_c[:, :, None] * x,
                               rtol=1e-10, atol=1e-12)


def pin_channels(M):
    rng = np.random.default_rng(15)
    x, delta, A, Bm, Cm = _inputs(rng, 2, 6, 5, 3)
    full = M.cycle_scan(x, delta, A, Bm, Cm, 3)
    np.testing.assert_allclose(M.cycle_scan_channels(x, delta, A, Bm, Cm, [4, 1], 3), full[:, :, [4, 1]],
                               rtol=1e-13, atol=1e-13)


PINS = [pin_golden, pin_zoh_van_loan, pin_scan_matrix_form, pin_cycle_matrix_form, pin_cycle_properties, pin_channels]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(C)


_orig_zoh = C.zoh
_orig_scan = C.selective_scan
_orig_cycle = C.cycle_scan


def _zoh_euler(delta, a, b):
    abar, _ = _orig_zoh(delta, a, b)
    return abar, np.asarray(delta, dtype=np.float64)[..., None] * np.asarray(b, dtype=np.float64)


def _zoh_b_dropped(delta, a, b):
    return _orig_zoh(delta, a, np.ones_like(np.asarray(b, dtype=np.float64)))


def _zoh_decay_sign(delta, a, b):
    return _orig_zoh(delta, -np.asarray(a, dtype=np.float64), b)


def _scan_output_before_update(x, delta, A, Bm, Cm, h0=None):
    y, h = _orig_scan(x, delta, A, Bm, Cm, h0)
    # y_t = C_t . h_{t-1}: shift the state sequence by one token
    ys = np.zeros_like(y)
    hs = np.zeros((x.shape[0], x.shape[2], np.asarray(A).shape[1]))
    for t in range(x.shape[1]):
        ys[:, t, :] = np.einsum("bdn,bn->bd", hs, np.asarray(Cm, dtype=np.float64)[:, t, :])
        abar, bbar = _orig_zoh(np.asarray(delta, dtype=np.float64)[:, t, :], np.asarray(A)[None],
                               np.asarray(Bm, dtype=np.float64)[:, t, None, :])
        hs = abar * hs + bbar * np.asarray(x, dtype=np.float64)[:, t, :, None]
    return ys, hs


def _scan_b_c_swapped(x, delta, A, Bm, Cm, h0=None):
    return _orig_scan(x, delta, A, Cm, Bm, h0)


def _cycle_state_reset(x, delta, A, Bm, Cm, repeats=3):
    # each copy scanned from a zero state: the state does not run on into the next copy
    return repeats * _orig_scan(x, delta, A, Bm, Cm)[0]


def _cycle_one_copy(x, delta, A, Bm, Cm, repeats=3):
    return _orig_cycle(x, delta, A, Bm, Cm, 1)


MUTANTS = {
    "zoh_euler_hold": {"zoh": _zoh_euler},
    "zoh_b_dropped": {"zoh": _zoh_b_dropped},
    "zoh_decay_sign": {"zoh": _zoh_decay_sign},
    "scan_output_before_update": {"selective_scan": _scan_output_before_update},
    "scan_b_c_swapped": {"selective_scan": _scan_b_c_swapped},
    "cycle_state_reset": {"cycle_scan": _cycle_state_reset},
    "cycle_one_copy": {"cycle_scan": _cycle_one_copy},
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    for attr, fn in MUTANTS[name].items():
        monkeypatch.setattr(C, attr, fn)
    failed = []
    for pin in PINS:
        try:
            with np.errstate(over="ignore", invalid="ignore"):   # a wrong decay sign overflows
                pin(C)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, "mutant %s passed every pin" % name

"""Cycle-scan: a selective state-space scan over the token sequence repeated, fp64.

TEST INFRASTRUCTURE, NOT PRODUCT CODE (see the package docstring).

HRSAM's Cycle-scan module (Sec. 3.5) runs a state space model over the image tokens.  The
continuous system h'(t) = A h(t) + B x(t), y(t) = C h(t) is discretised with the zero-order
hold of step Delta (the SSM equations of Sec. 3.5):

    h_t = Abar h_{t-1} + Bbar x_t,   y_t = C h_t,
    Abar = exp(Delta A),   Bbar = (Delta A)^{-1} (exp(Delta A) - I) Delta B.

The paper uses the selective form of Mamba, which it cites for the details: every channel
of a d-channel sequence is scanned on its own, with a diagonal A of N entries per channel,
and Delta (per token and channel), B and C (per token, N entries, shared by the channels)
given as inputs.  For a diagonal A the hold is entry-wise:
Abar[n] = exp(Delta a[n]) and Bbar[n] = (exp(Delta a[n]) - 1) / a[n] * b[n].

Cycle-scan repeats the token sequence r = 3 times, one copy after the other, scans the
3L tokens in that order (the state runs on from one copy into the next), splits the output
into the r copies and sums them.  A repeated token is the same token, so its Delta, B and C
repeat with it.

Layouts: x, delta, y [batch, L, d]; A [d, N]; Bm, Cm [batch, L, N].
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def zoh(delta, a, b):
    """Zero-order hold of one step for a diagonal A: (Abar, Bbar) for step delta [...],
    diagonal a [..., N] and input vector b [..., N] (broadcast).  a = 0 takes the limit
    Bbar = delta * b."""
    delta, a, b = _f64(delta), _f64(a), _f64(b)
    da = delta[..., None] * a
    abar = np.exp(da)
    with np.errstate(divide="ignore", invalid="ignore"):
        bbar = np.where(a != 0.0, np.expm1(da) / np.where(a != 0.0, a, 1.0) * b, delta[..., None] * b)
    return abar, bbar


def selective_scan(x, delta, A, Bm, Cm, h0=None):
    """The discretised SSM over one sequence per channel, in token order.
    x, delta [batch, L, d]; A [d, N]; Bm, Cm [batch, L, N]; h0 [batch, d, N] or None (zeros).
    Returns (y [batch, L, d], final state [batch, d, N])."""
    x, delta, A, Bm, Cm = _f64(x), _f64(delta), _f64(A), _f64(Bm), _f64(Cm)
    nb, L, d = x.shape
    h = np.zeros((nb, d, A.shape[1])) if h0 is None else _f64(h0).copy()
    y = np.empty((nb, L, d))
    for t in range(L):
        abar, bbar = zoh(delta[:, t, :], A[None, :, :], Bm[:, t, None, :])   # [batch, d, N]
        h = abar * h + bbar * x[:, t, :, None]
        y[:, t, :] = np.einsum("bdn,bn->bd", h, Cm[:, t, :])
    return y, h


def cycle_scan(x, delta, A, Bm, Cm, repeats=3):
    """Cycle-scan by its definition: the sequence and its per-token Delta, B, C laid out
    `repeats` times one after the other, scanned once from a zero state, the output cut
    back into the copies and summed."""
    x, delta, Bm, Cm = _f64(x), _f64(delta), _f64(Bm), _f64(Cm)
    L = x.shape[1]
    rep = lambda a: np.concatenate([a] * repeats, axis=1)
    y_long, _ = selective_scan(rep(x), rep(delta), A, rep(Bm), rep(Cm))
    return sum(y_long[:, k * L:(k + 1) * L, :] for k in range(repeats))


def cycle_scan_channels(x, delta, A, Bm, Cm, channels, repeats=3):
    """cycle_scan restricted to some channels (the channels are independent): y[:, :, channels]."""
    ch = np.asarray(channels)
    return cycle_scan(_f64(x)[:, :, ch], _f64(delta)[:, :, ch], _f64(A)[ch], Bm, Cm, repeats)

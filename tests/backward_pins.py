"""Pins of the fp64 backward oracle (``oracle.backward``): checks against facts that do not
come from the backward code itself.

Each ``pin_*`` takes the backward module (so the mutation tests can hand in a patched copy)
and raises AssertionError when the oracle disagrees with:

* central finite differences of the loss sum(dout * out), where out comes from the
  single-grid textbook forward (explicit roll, pad, partition and masked softmax -- none of
  the backward's region code): a random direction through every input at once, and single
  coordinates at the grid corners and on the pad token;
* library autograd: window >= grid with no shift is global attention, whose gradients
  PyTorch's float64 scaled_dot_product_attention backward gives;
* closed forms: constant v makes the output independent of q and k (dq = dk = 0); softmax
  rows sum to one, so the dv rows sum to the dout rows; adding one vector to every key a
  query sees leaves its output unchanged, so dk sums to zero over each region (MASK) and
  over all rows (KV-token);
* the log-sum-exp read off the textbook forward with one-hot values: out[i, j] is then the
  attention probability P_ij, and LSE_i = z_ij + log w_j - log P_ij; in the global case,
  scipy's logsumexp.
"""
from __future__ import annotations

import math

import numpy as np
import scipy.special
import torch
import torch.nn.functional as F

from oracle import swin_oracle as FWD
from oracle import multiscale as MS

# (H, W, window, shift, pad_mode): ragged grids, every shift class, both padding modes
CASES = [
    (6, 5, 4, 2, 0), (6, 5, 4, 2, 1), (7, 9, 4, 1, 0), (7, 9, 4, 3, 1),
    (5, 5, 3, 0, 0), (5, 5, 3, 0, 1), (4, 7, 8, 5, 1), (8, 8, 4, 0, 1),
]


def _inputs(rng, B, L, heads, d, pad_mode):
    extra = 1 if pad_mode == FWD.PAD_KVTOKEN else 0
    return (rng.standard_normal((B, L, heads, d)), rng.standard_normal((B, L + extra, heads, d)),
            rng.standard_normal((B, L + extra, heads, d)), rng.standard_normal((B, L, heads, d)))


def _loss(q, k, v, dout, H, W, window, shift, pad_mode):
    return float((dout * FWD.swin_attention_textbook(q, k, v, H, W, window, shift, pad_mode)).sum())


def pin_directional_fd(B):
    rng = np.random.default_rng(11)
    for H, W, k, s, pm in CASES:
        q, kk, v, do = _inputs(rng, 2, H * W, 2, 4, pm)
        dq, dk, dv = B.swin_attention_bwd(q, kk, v, do, H, W, k, s, pm)
        U = [rng.standard_normal(x.shape) for x in (q, kk, v)]
        h = 1e-5
        f = lambda t: _loss(q + t * U[0], kk + t * U[1], v + t * U[2], do, H, W, k, s, pm)
        fd = (f(h) - f(-h)) / (2 * h)
        an = float((dq * U[0]).sum() + (dk * U[1]).sum() + (dv * U[2]).sum())
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), ((H, W, k, s, pm), fd, an)


def pin_coordinate_fd(B):
    rng = np.random.default_rng(12)
    for H, W, k, s, pm in CASES[:4]:
        q, kk, v, do = _inputs(rng, 1, H * W, 1, 4, pm)
        grads = B.swin_attention_bwd(q, kk, v, do, H, W, k, s, pm)
        rows = [0, W - 1, (H - 1) * W, H * W - 1] + ([H * W] if pm else [])
        for which, g in enumerate(grads):
            for r in rows:
                if which == 0 and r >= H * W:
                    continue
                for ch in (0, 3):
                    args = [q, kk, v]
                    e = np.zeros_like(args[which])
                    e[0, r, 0, ch] = 1.0
                    h = 1e-5
                    plus = [a + h * e if i == which else a for i, a in enumerate(args)]
                    minus = [a - h * e if i == which else a for i, a in enumerate(args)]
                    fd = (_loss(*plus, do, H, W, k, s, pm) - _loss(*minus, do, H, W, k, s, pm)) / (2 * h)
                    assert abs(fd - g[0, r, 0, ch]) <= 1e-7 * max(1.0, abs(fd)), \
                        ((H, W, k, s, pm), "qkv"[which], r, ch, fd, g[0, r, 0, ch])


def pin_global_autograd(B):
    rng = np.random.default_rng(13)
    for H, W, d in ((3, 4, 8), (5, 5, 4)):
        q, kk, v, do = _inputs(rng, 2, H * W, 3, d, 0)
        dq, dk, dv = B.swin_attention_bwd(q, kk, v, do, H, W, max(H, W) + 1, 0, 0)
        t = [torch.tensor(x.transpose(0, 2, 1, 3).copy(), requires_grad=True) for x in (q, kk, v)]
        o = F.scaled_dot_product_attention(*t)
        o.backward(torch.from_numpy(do.transpose(0, 2, 1, 3).copy()))
        for mine, ref in zip((dq, dk, dv), t):
            np.testing.assert_allclose(mine, ref.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)


def pin_constant_values(B):
    rng = np.random.default_rng(14)
    for H, W, k, s, pm in CASES:
        q, kk, v, do = _inputs(rng, 1, H * W, 2, 4, pm)
        v = np.broadcast_to(rng.standard_normal((1, 1, 2, 4)), v.shape).copy()
        dq, dk, dv = B.swin_attention_bwd(q, kk, v, do, H, W, k, s, pm)
        assert np.abs(dq).max() < 1e-12 and np.abs(dk).max() < 1e-12, (H, W, k, s, pm)
        np.testing.assert_allclose(dv.sum(axis=1), do.sum(axis=1), rtol=1e-12, atol=1e-12)


def pin_row_sums_and_key_translation(B):
    rng = np.random.default_rng(15)
    for H, W, k, s, pm in CASES:
        q, kk, v, do = _inputs(rng, 1, H * W, 2, 4, pm)
        dq, dk, dv = B.swin_attention_bwd(q, kk, v, do, H, W, k, s, pm)
        np.testing.assert_allclose(dv.sum(axis=1), do.sum(axis=1), rtol=1e-11, atol=1e-11)
        if pm == FWD.PAD_KVTOKEN:
            assert np.abs(dk.sum(axis=1)).max() < 1e-11, (H, W, k, s, pm)
            continue
        # MASK: regions cut from first principles (not the oracle's region helper)
        ry = _labels(H, k, s)
        rx = _labels(W, k, s)
        for a in np.unique(ry):
            for b in np.unique(rx):
                rows = [y * W + x for y in range(H) for x in range(W) if ry[y] == a and rx[x] == b]
                assert np.abs(dk[:, rows].sum(axis=1)).max() < 1e-11, (H, W, k, s, a, b)


def _labels(n, k, s):
    """Region of each coordinate from first principles: cut the axis at s, s + k, s + 2k, ..."""
    cuts = [c for c in range(s, n, k) if c > 0]
    return np.searchsorted(np.array(cuts + [n + 1]), np.arange(n), side="right")


def pin_lse_one_hot(B):
    rng = np.random.default_rng(16)
    for H, W, k, s, pm in CASES:
        L = H * W
        d = L + 1
        q, kk, _, _ = _inputs(rng, 1, L, 1, d, pm)
        v = np.zeros_like(kk)
        v[0, np.arange(v.shape[1]), 0, np.arange(v.shape[1])] = 1.0     # value of key j = e_j
        out = FWD.swin_attention_textbook(q, kk, v, H, W, k, s, pm)      # out[i, j] = P_ij
        lse = B.swin_attention_lse(q, kk, v, H, W, k, s, pm)
        c = 1.0 / math.sqrt(d)
        for i in range(L):
            j = int(np.argmax(out[0, i, 0]))
            w = 1.0
            if j == L:
                w = float(k * k - np.count_nonzero(out[0, i, 0, :L] > 0))
            z = c * float(q[0, i, 0] @ kk[0, j, 0])
            want = z + math.log(w) - math.log(out[0, i, 0, j])
            assert abs(lse[0, 0, i] - want) < 1e-10, ((H, W, k, s, pm), i, lse[0, 0, i], want)


def pin_lse_global(B):
    rng = np.random.default_rng(17)
    H, W, d = 4, 6, 8
    q, kk, v, _ = _inputs(rng, 2, H * W, 3, d, 0)
    lse = B.swin_attention_lse(q, kk, v, H, W, 7, 0, 0)
    z = np.einsum("bihd,bjhd->bhij", q, kk) / math.sqrt(d)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=-1), rtol=1e-12, atol=1e-12)


def pin_ms_composition(B):
    """Multi-scale gradients equal finite differences of the multi-scale composition forward."""
    rng = np.random.default_rng(18)
    for grids, k, s, pm in ((((6, 5), (3, 4)), 4, 2, 1), (((5, 7), (2, 2), (4, 3)), 3, 1, 0)):
        L = sum(h * w for h, w in grids)
        q, kk, v, do = _inputs(rng, 1, L, 2, 4, pm)
        dq, dk, dv = B.swin_attention_ms_bwd(q, kk, v, do, grids, k, s, pm)
        U = [rng.standard_normal(x.shape) for x in (q, kk, v)]
        f = lambda t: float((do * MS.swin_attention_ms(q + t * U[0], kk + t * U[1], v + t * U[2],
                                                      grids, k, s, pm)).sum())
        h = 1e-5
        fd = (f(h) - f(-h)) / (2 * h)
        an = float((dq * U[0]).sum() + (dk * U[1]).sum() + (dv * U[2]).sum())
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (grids, fd, an)
        lse = B.swin_attention_ms_lse(q, kk, v, grids, k, s, pm)
        off = 0
        for h_, w_ in grids:
            rows = slice(off, off + h_ * w_)
            kg = np.concatenate([kk[:, rows], kk[:, L:]], axis=1) if pm else kk[:, rows]
            np.testing.assert_allclose(lse[:, :, rows],
                                       B.swin_attention_lse(q[:, rows], kg, kg, h_, w_, k, s, pm),
                                       rtol=1e-13, atol=1e-13)
            off += h_ * w_


PINS = [pin_directional_fd, pin_coordinate_fd, pin_global_autograd, pin_constant_values,
        pin_row_sums_and_key_translation, pin_lse_one_hot, pin_lse_global, pin_ms_composition]

"""Backward pass of Flash Swin attention, fp64.

TEST INFRASTRUCTURE, NOT PRODUCT CODE (see the package docstring).

The paper trains HRSAM through Flash Swin attention (App. D); the backward of Eq. 1 inside
each shifted window follows from the chain rule alone.  For one query i with key set R_i
(its region of Sec. 3.3; in KV-token mode, Sec. 3.4 / App. B, also the pad token p with
multiplicity m_i = window^2 - |R_i|), scale c = 1/sqrt(d), weights w_j = 1 (j in R_i) and
w_p = m_i:

    z_j   = c <q_i, k_j>
    LSE_i = log sum_l w_l exp(z_l)
    P_j   = w_j exp(z_j - LSE_i)                 (the weighted softmax of Eq. 1)
    o_i   = sum_j P_j v_j

Given dO_i = dLoss/do_i, with D_i = <dO_i, o_i>:

    dv_j += P_j dO_i
    dz_j  = P_j (<dO_i, v_j> - D_i)
    dq_i  = c sum_j dz_j k_j
    dk_j += c dz_j q_i

(sums over the weighted key set; the pad token's terms carry m_i through P_p).  Every query
of a region has the same key set, so the functions below work region by region.
``swin_attention_lse`` returns LSE_i, which a training forward stores for the backward.
"""
from __future__ import annotations

import math

import numpy as np

from .multiscale import _check_ms, _grids, grid_offsets
from .swin_oracle import PAD_KVTOKEN, _check, _f64, _region


def _key_sets(H, W, window, shift):
    """{region id: raster indices of its tokens} for the region rule of Sec. 3.3."""
    ry = _region(np.arange(H), window, shift)
    rx = _region(np.arange(W), window, shift)
    members = {}
    for y in range(H):
        for x in range(W):
            members.setdefault((int(ry[y]), int(rx[x])), []).append(y * W + x)
    return {r: np.array(m) for r, m in members.items()}


def _weighted_probs(z, w):
    """P = w exp(z - LSE) and LSE over the last axis, computed stably."""
    zm = z.max(axis=-1, keepdims=True)
    e = w * np.exp(z - zm)
    s = e.sum(axis=-1, keepdims=True)
    return e / s, (zm + np.log(s))[..., 0]


def _region_keys(q, k, v, keys, L, window, pad_mode):
    """Keys, values and weights one region's queries attend to: [B, m, h, d] x2, [m]."""
    kk, vk = k[:, keys], v[:, keys]
    w = np.ones(len(keys))
    if pad_mode == PAD_KVTOKEN:
        kk = np.concatenate([kk, k[:, L][:, None]], axis=1)
        vk = np.concatenate([vk, v[:, L][:, None]], axis=1)
        w = np.concatenate([w, [float(window * window - len(keys))]])
    return kk, vk, w


def _region_grads(qs, kk, vk, w, dos, c):
    """Gradients of one region: qs/dos [B, n, h, d] queries and upstream gradients, kk/vk
    [B, m, h, d] weighted keys and values.  Returns dq [B, n, h, d], dk and dv [B, m, h, d]."""
    z = c * np.einsum("bihd,bjhd->bhij", qs, kk)
    P, _ = _weighted_probs(z, w)
    o = np.einsum("bhij,bjhd->bihd", P, vk)
    D = np.einsum("bihd,bihd->bhi", dos, o)
    dP = np.einsum("bihd,bjhd->bhij", dos, vk)
    dz = P * (dP - D[..., None])
    dq = c * np.einsum("bhij,bjhd->bihd", dz, kk)
    dk = c * np.einsum("bhij,bihd->bjhd", dz, qs)
    dv = np.einsum("bhij,bihd->bjhd", P, dos)
    return dq, dk, dv


def swin_attention_lse(q, k, v, H, W, window, shift, pad_mode=0):
    """LSE_i of every query: [B, heads, L] float64, natural log of the (weighted) softmax
    denominator over the logits c <q_i, k_j>."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, heads, d = _check(q, k, v, H, W, window, shift, pad_mode)
    L = H * W
    c = 1.0 / math.sqrt(d)
    lse = np.empty((B, heads, L))
    for keys in _key_sets(H, W, window, shift).values():
        kk, _, w = _region_keys(q, k, v, keys, L, window, pad_mode)
        z = c * np.einsum("bihd,bjhd->bhij", q[:, keys], kk)
        lse[:, :, keys] = _weighted_probs(z, w)[1]
    return lse


def swin_attention_bwd(q, k, v, dout, H, W, window, shift, pad_mode=0):
    """(dq, dk, dv) for the upstream gradient dout [B, L, heads, d].  dk and dv have the
    shape of k and v; in KV-token mode their row L is the pad token's gradient, summed over
    every query that attends to it."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, heads, d = _check(q, k, v, H, W, window, shift, pad_mode)
    if dout.shape != q.shape:
        raise ValueError("dout must have the shape of q")
    L = H * W
    c = 1.0 / math.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for keys in _key_sets(H, W, window, shift).values():
        kk, vk, w = _region_keys(q, k, v, keys, L, window, pad_mode)
        gq, gk, gv = _region_grads(q[:, keys], kk, vk, w, dout[:, keys], c)
        n = len(keys)
        dq[:, keys] = gq
        dk[:, keys] += gk[:, :n]
        dv[:, keys] += gv[:, :n]
        if pad_mode == PAD_KVTOKEN:
            dk[:, L] += gk[:, n]
            dv[:, L] += gv[:, n]
    return dq, dk, dv


def _ms_slices(grids):
    offs, L = grid_offsets(grids)
    for (h, w), o in zip(_grids(grids), offs):
        yield h, w, slice(o, o + h * w), L


def _with_pad(x, rows, L, pad_mode):
    return np.concatenate([x[:, rows], x[:, L:L + 1]], axis=1) if pad_mode == PAD_KVTOKEN else x[:, rows]


def swin_attention_ms_lse(q, k, v, grids, window, shift, pad_mode=0):
    """Multi-scale LSE (App. C): each grid's queries over that grid's region, the pad token
    shared.  [B, heads, sum(H*W)]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    _check_ms(q, k, v, grids, pad_mode)
    out = np.empty((q.shape[0], q.shape[2], q.shape[1]))
    for h, w, rows, L in _ms_slices(grids):
        out[:, :, rows] = swin_attention_lse(q[:, rows], _with_pad(k, rows, L, pad_mode),
                                             _with_pad(v, rows, L, pad_mode), h, w, window, shift,
                                             pad_mode)
    return out


def swin_attention_ms_bwd(q, k, v, dout, grids, window, shift, pad_mode=0):
    """Multi-scale backward by composition: every grid's rows through ``swin_attention_bwd``;
    in KV-token mode the shared pad row's gradient is the sum over the grids."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    _check_ms(q, k, v, grids, pad_mode)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for h, w, rows, L in _ms_slices(grids):
        gq, gk, gv = swin_attention_bwd(q[:, rows], _with_pad(k, rows, L, pad_mode),
                                        _with_pad(v, rows, L, pad_mode), dout[:, rows], h, w,
                                        window, shift, pad_mode)
        n = h * w
        dq[:, rows] = gq
        dk[:, rows] = gk[:, :n]
        dv[:, rows] = gv[:, :n]
        if pad_mode == PAD_KVTOKEN:
            dk[:, L] += gk[:, n]
            dv[:, L] += gv[:, n]
    return dq, dk, dv

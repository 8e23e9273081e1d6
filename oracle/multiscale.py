"""Multi-scale Flash Swin attention (HRSAM++, Sec. 3.6 'Multi-scale attention', App. C), fp64.

TEST INFRASTRUCTURE, NOT PRODUCT CODE (see the package docstring).

The input holds the tokens of several grids one after the other (each grid row-major; the
paper's case is the image grid followed by the anchor-map grid).  Each grid gets its own
shifted-window attention: windows never span two grids.  In KV-token mode a single pad
token, the row after the last grid's tokens, is shared by every grid (App. C, KV-only
padding index mapping).

Three forms, written independently of each other:
  * ``swin_attention_ms``      -- by composition: the single-grid textbook form (explicit
                                  roll, pad, partition, masked softmax) on each grid's rows;
  * ``swin_attention_ms_fla``  -- App. C's index lists: the per-grid mappings of App. A/B
                                  concatenated with the grid's row offset, the pad index of
                                  every grid redirected to the shared last row, then
                                  block-diagonal attention and the inverse reorder;
  * ``swin_attention_ms_at``   -- brute force per query from the region rule within its grid.
"""
from __future__ import annotations

import math

import numpy as np

from .swin_oracle import (PAD_KVTOKEN, PAD_MASK, _f64, _softmax_weighted, _region,
                          fla_kv_padding_indices, fla_shift_window_indices,
                          swin_attention_textbook, window_sizes)


def _grids(grids):
    g = [(int(h), int(w)) for h, w in grids]
    if not g or any(h < 1 or w < 1 for h, w in g):
        raise ValueError("grids must be a non-empty list of (H, W) with H, W >= 1")
    return g


def grid_offsets(grids):
    """Row offset of each grid's first token, and the total token count."""
    g = _grids(grids)
    offs = np.concatenate([[0], np.cumsum([h * w for h, w in g])]).astype(np.int64)
    return offs[:-1], int(offs[-1])


def _check_ms(q, k, v, grids, pad_mode):
    if pad_mode not in (PAD_MASK, PAD_KVTOKEN):
        raise ValueError("pad_mode must be 0 (mask) or 1 (KV token)")
    _, L = grid_offsets(grids)
    if q.ndim != 4 or q.shape[1] != L:
        raise ValueError("q must be [B, sum(H*W), heads, d]")
    kv_rows = L + (1 if pad_mode == PAD_KVTOKEN else 0)
    if k.shape != (q.shape[0], kv_rows) + q.shape[2:] or v.shape != k.shape:
        raise ValueError("k, v must be [B, %d, heads, d]" % kv_rows)
    return q.shape[0], q.shape[2], q.shape[3]


def swin_attention_ms(q, k, v, grids, window, shift, pad_mode=PAD_MASK):
    """By composition: every grid on its own rows with the single-grid textbook form."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    _check_ms(q, k, v, grids, pad_mode)
    offs, L = grid_offsets(grids)
    out = np.empty_like(q)
    for (h, w), o in zip(_grids(grids), offs):
        rows = slice(o, o + h * w)
        if pad_mode == PAD_KVTOKEN:
            kg = np.concatenate([k[:, rows], k[:, L:L + 1]], axis=1)
            vg = np.concatenate([v[:, rows], v[:, L:L + 1]], axis=1)
        else:
            kg, vg = k[:, rows], v[:, rows]
        out[:, rows] = swin_attention_textbook(q[:, rows], kg, vg, h, w, window, shift, pad_mode)
    return out


def ms_shift_window_indices(grids, k, s):
    """App. C non-padding mapping: each grid's App. A list shifted by the grid's row offset,
    concatenated in grid order; lengths concatenated; ``inv`` restores the token order."""
    offs, _ = grid_offsets(grids)
    idx, lens = [], []
    for (h, w), o in zip(_grids(grids), offs):
        i, l, _ = fla_shift_window_indices(h, w, k, s)
        idx.append(i + o)
        lens.append(l)
    indices = np.concatenate(idx)
    return indices, np.concatenate(lens), np.argsort(indices, kind="stable")


def ms_kv_padding_indices(grids, k, s):
    """App. C KV-only padding mapping: each grid's App. B list (its pad slots point at its
    own row h*w) with real entries shifted by the grid's offset and pad entries sent to the
    shared pad row, the one after all grids."""
    offs, L = grid_offsets(grids)
    idx, lens = [], []
    for (h, w), o in zip(_grids(grids), offs):
        i, l = fla_kv_padding_indices(h, w, k, s)
        idx.append(np.where(i == h * w, L, i + o))
        lens.append(l)
    return np.concatenate(idx), np.concatenate(lens)


def swin_attention_ms_fla(q, k, v, grids, window, shift, pad_mode=PAD_MASK):
    """App. C form: reorder by the concatenated index list, block-diagonal attention,
    inverse reorder (KV-token mode: K/V gathered by the padding list, k*k per segment)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    _, _, d = _check_ms(q, k, v, grids, pad_mode)
    indices, lengths, inv = ms_shift_window_indices(grids, window, shift)
    if pad_mode == PAD_KVTOKEN:
        kv_idx, kv_len = ms_kv_padding_indices(grids, window, shift)
    else:
        kv_idx, kv_len = indices, lengths
    qI, kI, vI = q[:, indices], k[:, kv_idx], v[:, kv_idx]
    qs = np.concatenate([[0], np.cumsum(lengths)])
    ks = np.concatenate([[0], np.cumsum(kv_len)])
    Y = np.empty_like(qI)
    scale = 1.0 / math.sqrt(d)
    for i in range(len(lengths)):
        Qi = qI[:, qs[i]:qs[i + 1]].transpose(0, 2, 1, 3)
        Ki = kI[:, ks[i]:ks[i + 1]].transpose(0, 2, 1, 3)
        Vi = vI[:, ks[i]:ks[i + 1]].transpose(0, 2, 1, 3)
        z = np.matmul(Qi, np.swapaxes(Ki, -1, -2)) * scale
        p = np.exp(z - z.max(axis=-1, keepdims=True))
        p /= p.sum(axis=-1, keepdims=True)
        Y[:, qs[i]:qs[i + 1]] = np.matmul(p, Vi).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(Y[:, inv])


def swin_attention_ms_at(q, k, v, grids, window, shift, pad_mode, queries):
    """Brute force on selected queries [S, 4] of (b, grid, y, x): each query scans every
    token of its grid and keeps its region; KV-token mode adds the shared pad row with
    multiplicity k*k - (region size).  Returns [S, heads, d]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    _, heads, d = _check_ms(q, k, v, grids, pad_mode)
    g = _grids(grids)
    offs, L = grid_offsets(grids)
    scale = 1.0 / math.sqrt(d)
    queries = np.asarray(queries, dtype=np.int64).reshape(-1, 4)
    out = np.empty((len(queries), heads, d))
    for n, (b, gi, y, x) in enumerate(queries):
        h, w = g[gi]
        ry, rx = _region(np.arange(h), window, shift), _region(np.arange(w), window, shift)
        sel = (np.repeat(ry, w) == ry[y]) & (np.tile(rx, h) == rx[x])
        keys = offs[gi] + np.nonzero(sel)[0]
        qv = q[b, offs[gi] + y * w + x]
        z = np.einsum("hd,mhd->hm", qv, k[b, keys]) * scale
        wts = np.ones_like(z)
        vals = v[b, keys]
        if pad_mode == PAD_KVTOKEN:
            z = np.concatenate([z, (np.einsum("hd,hd->h", qv, k[b, L]) * scale)[:, None]], axis=1)
            wts = np.concatenate([wts, np.full((heads, 1), float(window * window - len(keys)))], axis=1)
            vals = np.concatenate([vals, v[b, L][None]], axis=0)
        out[n] = np.einsum("hm,mhd->hd", _softmax_weighted(z, wts), vals)
    return out


def ms_work_counts(B, heads, grids, head_dim, window, shift, pad_mode, elem_bytes):
    """Algorithmic FLOP and bytes of one multi-scale layer: the single-grid counts summed
    over the grids, with one shared pad row (KV-token mode) instead of one per grid."""
    pairs = 0.0
    for h, w in _grids(grids):
        n = window_sizes(h, w, window, shift).astype(np.float64)
        pairs += float((n * n).sum())
        if pad_mode == PAD_KVTOKEN:
            pairs += float((n * (n < window * window)).sum())
    _, L = grid_offsets(grids)
    rows = 4.0 * L + (2.0 if pad_mode == PAD_KVTOKEN else 0.0)
    return 4.0 * head_dim * heads * B * pairs, rows * B * heads * head_dim * elem_bytes

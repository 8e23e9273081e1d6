"""fp64 CPU oracle for Flash Swin attention — TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this module.  It shares nothing with the HIP library.

What is computed (HRSAM, arXiv 2407.02109):

* Eq. 1 (Sec. 3.2): scaled dot-product attention, one softmax per query.  The scale is
  ``1/sqrt(head_dim)`` per head (reading of Eq. 1's ``sqrt(C)`` for the multi-head case).
* Sec. 3.3 "Shift window" + App. A: Swin windows of size ``k`` shifted by ``s``.  The
  paper pads ``k - s`` virtual tokens in front of each axis and partitions the padded
  canvas into ``k x k`` windows; virtual tokens are dropped from the query and key sets.
  Equivalently (checked by the tests) token ``c`` of an axis belongs to region
  ``floor((c - s) / k)``, and a query attends to every real token of its region.
* Sec. 3.4 "KV-only padding" + App. B: every virtual key slot of a window reads one
  extra learnable K/V token stored at row ``L = H*W``; the key set of a window then has
  exactly ``k*k`` entries (the pad token counted once per virtual slot), queries are
  never padded.

Layout of every tensor argument: ``[B, L, heads, head_dim]`` with ``L = H*W`` tokens in
raster order (Sec. 3.3's vanilla map: token ``j`` sits at row ``j // W``, column
``j % W``).  In KV-token mode ``k`` and ``v`` carry ``L + 1`` rows, the last one being
the pad token.  All arithmetic is float64; inputs are converted exactly.

Four forms, each written independently from the paper:

(i)   ``swin_attention_textbook`` -- Plain Swin: pad to a multiple of k, cyclic shift by
      -s, partition, region mask + pad-key mask, softmax, P.V, reverse partition, shift
      back, crop.  This is the conventional implementation the paper compares against.
(ii)  ``swin_attention_canvas`` -- the paper's own construction: translate the grid by
      ``k - s`` virtual rows/cols, unshifted windows on the padded canvas, virtual keys
      masked (or filled with the pad token, one copy per slot), crop.
(iii) ``swin_attention_fla`` -- the FLA form: index mapping I, per-window lengths,
      block-diagonal attention on the reordered sequence, inverse mapping.
(iv)  ``swin_attention_bruteforce`` / ``swin_attention_at`` -- per query, straight from
      the region definition.
"""
from __future__ import annotations

import math

import numpy as np

PAD_MASK = 0      # virtual / out-of-grid key slots are excluded from the softmax
PAD_KVTOKEN = 1   # virtual key slots read the learnable token at row L (Sec. 3.4, App. B)


# ----------------------------------------------------------------------------------------
# shared input handling (no attention arithmetic)
# ----------------------------------------------------------------------------------------
def _check(q, k, v, H, W, window, shift, pad_mode):
    if q.ndim != 4:
        raise ValueError("q must be [B, L, heads, head_dim]")
    B, L, heads, d = q.shape
    if L != H * W:
        raise ValueError("q has %d rows, grid is %dx%d" % (L, H, W))
    want = L + 1 if pad_mode == PAD_KVTOKEN else L
    for name, t in (("k", k), ("v", v)):
        if t.shape != (B, want, heads, d):
            raise ValueError("%s must be [B, %d, heads, head_dim], got %s" % (name, want, t.shape))
    if window < 1 or not (0 <= shift < window):
        raise ValueError("need window >= 1 and 0 <= shift < window")
    if pad_mode not in (PAD_MASK, PAD_KVTOKEN):
        raise ValueError("pad_mode must be 0 or 1")
    return B, heads, d


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _softmax_weighted(logits, weights):
    """Softmax over the last axis where key j counts ``weights[..., j]`` times.

    ``weights`` is 0 for excluded keys.  Returns the normalised probabilities.
    Rows whose every weight is zero come back as NaN (they belong to padded queries that
    the callers crop away)."""
    with np.errstate(invalid="ignore", divide="ignore"):
        z = np.where(weights > 0, logits, -np.inf)
        m = z.max(axis=-1, keepdims=True)
        e = weights * np.exp(z - m)
        return e / e.sum(axis=-1, keepdims=True)


# ----------------------------------------------------------------------------------------
# (i) textbook Plain Swin: pad -> roll(-s) -> partition -> region mask -> softmax -> reverse
# ----------------------------------------------------------------------------------------
def _pad_bottom_right(x, Hp, Wp):
    """Zero-pad grid tensor [B, H, W, ...] to [B, Hp, Wp, ...]."""
    out = np.zeros((x.shape[0], Hp, Wp) + x.shape[3:], dtype=np.float64)
    out[:, : x.shape[1], : x.shape[2]] = x
    return out


def _cyclic_shift(x, s, axes):
    """Swin's cyclic shift: move the grid up/left by s (np.roll by -s)."""
    return np.roll(x, (-s, -s), axis=axes)


def _cyclic_unshift(x, s, axes):
    return np.roll(x, (s, s), axis=axes)


def _region_labels_1d(n, k, s):
    """Region label of each row (column) of the shifted, padded frame of length n.

    In the shifted frame every window [i*k, (i+1)*k) is one region, except the last one,
    which holds tokens wrapped round from the other border: its first k - s entries
    came from the end of the axis, its last s from the start.  Labels only need to differ
    inside a window, so three labels suffice (Swin's three slices)."""
    lab = np.zeros(n, dtype=np.int64)
    if s > 0:
        lab[n - k: n - s] = 1
        lab[n - s:] = 2
    return lab


def _partition(x, k):
    """[B, Hp, Wp, heads, d] -> [B, nW, heads, k*k, d], windows in raster order,
    tokens row-major inside a window (Eq. nonshift)."""
    B, Hp, Wp, heads, d = x.shape
    x = x.reshape(B, Hp // k, k, Wp // k, k, heads, d)
    x = x.transpose(0, 1, 3, 5, 2, 4, 6)
    return x.reshape(B, (Hp // k) * (Wp // k), heads, k * k, d)


def _partition_map(m, k):
    """[Hp, Wp] -> [nW, k*k], same order as ``_partition``."""
    Hp, Wp = m.shape
    return m.reshape(Hp // k, k, Wp // k, k).transpose(0, 2, 1, 3).reshape(-1, k * k)


def _unpartition(x, k, Hp, Wp):
    """Inverse of ``_partition``."""
    B, nW, heads, kk, d = x.shape
    x = x.reshape(B, Hp // k, Wp // k, heads, k, k, d)
    x = x.transpose(0, 1, 4, 2, 5, 3, 6)
    return x.reshape(B, Hp, Wp, heads, d)


def _pad_multiplicity(allowed):
    """Virtual key slots seen by each query of a window: its k*k slots minus the real
    keys of its own region (Sec. 3.4: they all read the one pad token)."""
    return allowed.shape[1] - allowed.sum(axis=1)


def _window_attention(qw, kw, vw, allowed, scale, kpad=None, vpad=None):
    """Attention inside one window.

    qw, kw, vw: [B, heads, n, d] with n = k*k slots; allowed: [n, n] bool (query, key).
    With a pad token (kpad, vpad: [B, heads, d]) every query also attends the pad token
    with multiplicity ``k*k - (number of keys it is allowed)``: the virtual slots of its
    own k x k window (Sec. 3.4)."""
    logits = np.matmul(qw, np.swapaxes(kw, -1, -2)) * scale          # [B, h, n, n]
    weights = np.broadcast_to(allowed.astype(np.float64), logits.shape)
    values = vw
    if kpad is not None:
        pad_count = _pad_multiplicity(allowed)                          # [n]
        zpad = np.einsum("bhnd,bhd->bhn", qw, kpad) * scale             # [B, h, n]
        logits = np.concatenate([logits, zpad[..., None]], axis=-1)
        wpad = np.broadcast_to(pad_count.astype(np.float64)[:, None], zpad.shape[:2] + (qw.shape[2], 1))
        weights = np.concatenate([weights, wpad], axis=-1)
        values = np.concatenate([vw, vpad[:, :, None, :]], axis=2)
    p = _softmax_weighted(logits, weights)
    return np.matmul(p, values)


def swin_attention_textbook(q, k, v, H, W, window, shift, pad_mode=PAD_MASK):
    """Form (i): conventional (Plain) shifted-window attention, explicit copies throughout.

    Steps: zero-pad bottom/right to a multiple of the window; cyclic shift by -shift;
    label the three Swin regions of the shifted frame; partition into windows; mask
    keys of another region and padded keys (-inf); softmax; P.V; reverse the partition;
    shift back by +shift; crop to H x W.

    KV-token mode (Sec. 3.4): every key slot of a query's k x k window that is not a
    real token of its region is filled by the pad token (row L of k and v).  In the
    shifted frame that count is k*k minus the query's allowed real keys."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, heads, d = _check(q, k, v, H, W, window, shift, pad_mode)
    kk, s = window, shift
    L = H * W
    Hp = -(-H // kk) * kk
    Wp = -(-W // kk) * kk
    scale = 1.0 / math.sqrt(d)

    def grid(x):
        return x[:, :L].reshape(B, H, W, heads, d)

    qp = _cyclic_shift(_pad_bottom_right(grid(q), Hp, Wp), s, (1, 2))
    kp = _cyclic_shift(_pad_bottom_right(grid(k), Hp, Wp), s, (1, 2))
    vp = _cyclic_shift(_pad_bottom_right(grid(v), Hp, Wp), s, (1, 2))
    valid = np.zeros((Hp, Wp), dtype=bool)
    valid[:H, :W] = True
    valid = _cyclic_shift(valid, s, (0, 1))
    labels = _region_labels_1d(Hp, kk, s)[:, None] * 3 + _region_labels_1d(Wp, kk, s)[None, :]

    qw, kw, vw = _partition(qp, kk), _partition(kp, kk), _partition(vp, kk)
    labw = _partition_map(labels, kk)
    validw = _partition_map(valid, kk)
    kpad = k[:, L] if pad_mode == PAD_KVTOKEN else None
    vpad = v[:, L] if pad_mode == PAD_KVTOKEN else None

    out_w = np.empty_like(qw)
    for wi in range(qw.shape[1]):
        allowed = (labw[wi][:, None] == labw[wi][None, :]) & validw[wi][None, :]
        out_w[:, wi] = _window_attention(qw[:, wi], kw[:, wi], vw[:, wi], allowed, scale, kpad, vpad)

    out = _cyclic_unshift(_unpartition(out_w, kk, Hp, Wp), s, (1, 2))
    return np.ascontiguousarray(out[:, :H, :W].reshape(B, L, heads, d))


# ----------------------------------------------------------------------------------------
# (ii) translate-canvas form: the paper's virtual-token padding (Sec. 3.3, App. A/B)
# ----------------------------------------------------------------------------------------
def _canvas_geometry(H, W, k, s):
    """Offset and size of the virtual-token canvas.

    The paper puts k - s virtual tokens in front of each axis (k/2 for s = k/2) so that
    unshifted k x k windows on the canvas are the shifted windows on the grid.  The back
    is padded up to a multiple of k (for the paper's s = k/2 and k | H this is the
    (H + k) x (W + k) canvas)."""
    o = (k - s) % k
    Hc = -(-(H + o) // k) * k
    Wc = -(-(W + o) // k) * k
    return o, Hc, Wc


def swin_attention_canvas(q, k, v, H, W, window, shift, pad_mode=PAD_MASK):
    """Form (ii): unshifted windows on the virtual-token canvas.

    MASK mode: virtual key slots are excluded.  KV-token mode: every virtual slot holds a
    copy of the pad token (row L), so each window has exactly k*k keys, repeated pad
    copies included (App. B's lengths)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, heads, d = _check(q, k, v, H, W, window, shift, pad_mode)
    kk, s = window, shift
    L = H * W
    o, Hc, Wc = _canvas_geometry(H, W, kk, s)
    scale = 1.0 / math.sqrt(d)

    def canvas(x, fill=None):
        c = np.zeros((B, Hc, Wc, heads, d))
        if fill is not None:
            c[:] = fill[:, None, None]
        c[:, o:o + H, o:o + W] = x[:, :L].reshape(B, H, W, heads, d)
        return c

    real = np.zeros((Hc, Wc), dtype=bool)
    real[o:o + H, o:o + W] = True
    if pad_mode == PAD_KVTOKEN:
        kc, vc = canvas(k, k[:, L]), canvas(v, v[:, L])
        key_ok = np.ones_like(real)
    else:
        kc, vc = canvas(k), canvas(v)
        key_ok = real
    qc = canvas(q)

    # unshifted window partition of the canvas, in the canvas' own raster order
    nwy, nwx = Hc // kk, Wc // kk
    out_c = np.full((B, Hc, Wc, heads, d), np.nan)
    for wy in range(nwy):
        for wx in range(nwx):
            ys = slice(wy * kk, wy * kk + kk)
            xs = slice(wx * kk, wx * kk + kk)
            qw = qc[:, ys, xs].reshape(B, kk * kk, heads, d).transpose(0, 2, 1, 3)
            kw = kc[:, ys, xs].reshape(B, kk * kk, heads, d).transpose(0, 2, 1, 3)
            vw = vc[:, ys, xs].reshape(B, kk * kk, heads, d).transpose(0, 2, 1, 3)
            ok = key_ok[ys, xs].reshape(-1).astype(np.float64)
            logits = np.matmul(qw, np.swapaxes(kw, -1, -2)) * scale
            p = _softmax_weighted(logits, np.broadcast_to(ok, logits.shape))
            ow = np.matmul(p, vw)                                       # [B, h, k*k, d]
            out_c[:, ys, xs] = ow.transpose(0, 2, 1, 3).reshape(B, kk, kk, heads, d)
    out = out_c[:, o:o + H, o:o + W]
    return np.ascontiguousarray(out.reshape(B, L, heads, d))


# ----------------------------------------------------------------------------------------
# (iii) FLA form: index mapping, lengths, block-diagonal attention, inverse mapping
# ----------------------------------------------------------------------------------------
def _canvas_coords(H, W, k, s):
    """The k*k slots of every canvas window, from the definitions of App. A.

    The canvas is the grid with o = (k - s) mod k virtual tokens in front of each axis and
    as many behind as make it a multiple of k (Sec. 3.3); its unshifted k x k windows are
    taken in raster order of the windows.  Window (wy, wx) covers grid rows
    wy*k - o .. wy*k - o + k - 1 and grid columns wx*k - o .. wx*k - o + k - 1; its slot
    (a, b), numbered row-major inside the window (Eq. nonshift on the extended domain),
    holds grid token (y, x) = (wy*k - o + a, wx*k - o + b), whose raster index is y*W + x,
    or is virtual (-1) when (y, x) lies outside the grid.  Returns [windows, k*k]."""
    o = (k - s) % k
    nwy = -(-(H + o) // k)
    nwx = -(-(W + o) // k)
    out = np.full((nwy * nwx, k * k), -1, dtype=np.int64)
    for wy in range(nwy):
        for wx in range(nwx):
            for a in range(k):
                y = wy * k - o + a
                for b in range(k):
                    x = wx * k - o + b
                    if 0 <= y < H and 0 <= x < W:
                        out[wy * nwx + wx, a * k + b] = y * W + x
    return out


def fla_shift_window_indices(H, W, k, s):
    """Shift-window index mapping of App. A (Eq. finalswin, Eq. finalswinlengths).

    Returns ``(indices, lengths, inv)``: ``indices`` lists the real tokens of window 0, then
    of window 1, ..., each window's in its own row-major order, so ``x[indices]`` puts the
    tokens of each window next to each other; ``lengths[i]`` is the number of real tokens of
    window i; ``inv`` is the inverse permutation (``inv[indices[j]] = j``), so
    ``x[indices][inv] == x``."""
    slots = _canvas_coords(H, W, k, s)
    per_window = [row[row >= 0] for row in slots]
    indices = np.concatenate(per_window)
    lengths = np.array([len(t) for t in per_window], dtype=np.int64)
    inv = np.empty(H * W, dtype=np.int64)
    inv[indices] = np.arange(len(indices), dtype=np.int64)
    return indices, lengths, inv


def fla_kv_padding_indices(H, W, k, s):
    """KV-only padding index mapping of App. B.

    Every slot of every canvas window is kept; virtual slots point at the pad token,
    row ``H*W``.  All lengths are k*k."""
    coords = _canvas_coords(H, W, k, s)
    flat = coords.reshape(-1).copy()
    flat[flat < 0] = H * W
    return flat, np.full(coords.shape[0], k * k, dtype=np.int64)


def swin_attention_fla(q, k, v, H, W, window, shift, pad_mode=PAD_MASK):
    """Form (iii): Reorder(X, I) -> block-diagonal attention -> Reorder(Y, I^-1) (Sec. 3.2).

    MASK mode: the K/V segments are the same as the Q segments.  KV-token mode: the K/V
    sequence is gathered with App. B's mapping (pad row repeated) and every K/V segment
    has k*k entries, while Q keeps App. A's segments (extended FLA, Sec. 3.4)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, heads, d = _check(q, k, v, H, W, window, shift, pad_mode)
    indices, lengths, inv = fla_shift_window_indices(H, W, window, shift)
    scale = 1.0 / math.sqrt(d)
    qI = q[:, indices]
    if pad_mode == PAD_KVTOKEN:
        kv_idx, kv_len = fla_kv_padding_indices(H, W, window, shift)
        kI, vI = k[:, kv_idx], v[:, kv_idx]
    else:
        kv_len = lengths
        kI, vI = k[:, indices], v[:, indices]
    q_starts = np.concatenate([[0], np.cumsum(lengths)])
    kv_starts = np.concatenate([[0], np.cumsum(kv_len)])
    Y = np.empty_like(qI)
    for i in range(len(lengths)):
        qs = slice(q_starts[i], q_starts[i + 1])
        ks = slice(kv_starts[i], kv_starts[i + 1])
        Qi = qI[:, qs].transpose(0, 2, 1, 3)                 # [B, h, n, d]
        Ki = kI[:, ks].transpose(0, 2, 1, 3)
        Vi = vI[:, ks].transpose(0, 2, 1, 3)
        z = np.matmul(Qi, np.swapaxes(Ki, -1, -2)) * scale
        z = z - z.max(axis=-1, keepdims=True)
        p = np.exp(z)
        p = p / p.sum(axis=-1, keepdims=True)
        Y[:, qs] = np.matmul(p, Vi).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(Y[:, inv])


# ----------------------------------------------------------------------------------------
# (iv) brute force from the region definition
# ----------------------------------------------------------------------------------------
def _region(c, k, s):
    """Region index of grid coordinate c: tokens c and c' share a window axis slot iff
    floor((c - s)/k) == floor((c' - s)/k)."""
    return np.floor_divide(np.asarray(c) - s, k)


def swin_attention_at(q, k, v, H, W, window, shift, pad_mode, queries):
    """Form (iv) on selected query tokens.

    queries: int array [S, 3] of (b, y, x).  Returns [S, heads, d] float64.  Each query
    scans all H*W keys and keeps those of its region; in KV-token mode the pad token
    is added with multiplicity k*k - (region size)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, heads, d = _check(q, k, v, H, W, window, shift, pad_mode)
    scale = 1.0 / math.sqrt(d)
    L = H * W
    ry = _region(np.arange(H), window, shift)
    rx = _region(np.arange(W), window, shift)
    tok_ry = np.repeat(ry, W)
    tok_rx = np.tile(rx, H)
    queries = np.asarray(queries, dtype=np.int64).reshape(-1, 3)
    out = np.empty((len(queries), heads, d))
    for n, (b, y, x) in enumerate(queries):
        keys = np.nonzero((tok_ry == ry[y]) & (tok_rx == rx[x]))[0]
        qv = q[b, y * W + x]                                    # [h, d]
        kv = k[b, keys]                                         # [m, h, d]
        vv = v[b, keys]
        z = np.einsum("hd,mhd->hm", qv, kv) * scale
        wts = np.ones_like(z)
        vals = vv
        if pad_mode == PAD_KVTOKEN:
            n_pad = window * window - len(keys)
            z = np.concatenate([z, (np.einsum("hd,hd->h", qv, k[b, L]) * scale)[:, None]], axis=1)
            wts = np.concatenate([wts, np.full((heads, 1), float(n_pad))], axis=1)
            vals = np.concatenate([vv, v[b, L][None]], axis=0)
        p = _softmax_weighted(z, wts)                           # [h, m]
        out[n] = np.einsum("hm,mhd->hd", p, vals)
    return out


def swin_attention_bruteforce(q, k, v, H, W, window, shift, pad_mode=PAD_MASK):
    """Form (iv) over every query token (tiny inputs only)."""
    B = np.asarray(q).shape[0]
    bb, yy, xx = np.meshgrid(np.arange(B), np.arange(H), np.arange(W), indexing="ij")
    queries = np.stack([bb.ravel(), yy.ravel(), xx.ravel()], axis=1)
    out = swin_attention_at(q, k, v, H, W, window, shift, pad_mode, queries)
    heads, d = out.shape[1:]
    return out.reshape(B, H * W, heads, d)


# ----------------------------------------------------------------------------------------
# work accounting (used by the benchmark to state algorithmic flops/bytes)
# ----------------------------------------------------------------------------------------
def window_sizes(H, W, window, shift):
    """Number of real tokens of every window (the FLA lengths), from the region map."""
    _, lengths, _ = fla_shift_window_indices(H, W, window, shift)
    return lengths


def work_counts(B, heads, H, W, head_dim, window, shift, pad_mode, elem_bytes):
    """Algorithmic FLOP and HBM bytes of one layer.

    FLOP: 2*d per (query, key) pair for Q.K^T and again for P.V, summed over the real
    pairs of every window (masked pairs are not counted); in KV-token mode one more key
    (the pad token) per query whose window has virtual slots.  Bytes: q, k, v read once
    and out written once (plus the pad rows)."""
    n = window_sizes(H, W, window, shift).astype(np.float64)
    pairs = float((n * n).sum())
    if pad_mode == PAD_KVTOKEN:
        pairs += float((n * (n < window * window)).sum())
    flops = 4.0 * head_dim * heads * B * pairs
    rows = 4.0 * H * W + (2.0 if pad_mode == PAD_KVTOKEN else 0.0)
    bytes_ = rows * B * heads * head_dim * elem_bytes
    return flops, bytes_

"""Rotary position embedding (RoPE) on q and k ahead of Flash Swin attention, fp64.

TEST INFRASTRUCTURE, NOT PRODUCT CODE (see the package docstring).

HRSAM replaces SAM's relative position bias with RoPE (Sec. 3.1, citing RoFormer) so that
attention keeps no O(N^2) bias and memory-efficient kernels apply.  The paper does not
spell out the 2-D variant; the reading taken here is the axial form of the ViTs it builds
on: a head of d channels is split in two halves, the first rotated by the token's row
coordinate and the second by its column coordinate.  Within a half of d/2 channels, the
channel pair (2j, 2j + 1) is the complex number x[2j] + i x[2j + 1], multiplied by
exp(i p theta^(-2j / (d/2))), where p = scale * (row or column index in the token grid)
and theta is the base (10000 in RoFormer).  The learnable pad token of KV-token mode has
no position and is not rotated.
"""
from __future__ import annotations

import numpy as np

from .swin_oracle import PAD_KVTOKEN, _f64, swin_attention_textbook


def rope_angles(H, W, d, theta=10000.0, scale=1.0, y0=0.0, x0=0.0):
    """Angle of every (token, channel pair): [H*W, d/2] float64.  Pairs 0 .. d/4-1 belong
    to the row half, pairs d/4 .. d/2-1 to the column half.  (y0, x0) shifts the
    coordinates (used by the tests)."""
    if d % 4:
        raise ValueError("head_dim must be a multiple of 4 for 2-D RoPE")
    half = d // 2
    j = np.arange(half // 2, dtype=np.float64)
    freq = float(theta) ** (-2.0 * j / half)
    ys = (np.arange(H, dtype=np.float64) + y0) * scale
    xs = (np.arange(W, dtype=np.float64) + x0) * scale
    row = np.repeat(ys, W)[:, None] * freq[None, :]
    col = np.tile(xs, H)[:, None] * freq[None, :]
    return np.concatenate([row, col], axis=1)


def apply_rope(x, H, W, theta=10000.0, scale=1.0, y0=0.0, x0=0.0, inverse=False):
    """Rotate the first H*W rows of x [B, rows, heads, d] (by the opposite angles when
    inverse: the transpose of the rotation); rows past H*W (the pad token) are returned
    unchanged."""
    x = _f64(x)
    B, rows, heads, d = x.shape
    L = H * W
    ang = rope_angles(H, W, d, theta, scale, y0, x0)          # [L, d/2]
    if inverse:
        ang = -ang
    c, s = np.cos(ang)[None, :, None, :], np.sin(ang)[None, :, None, :]
    out = x.copy()
    even, odd = x[:, :L, :, 0::2], x[:, :L, :, 1::2]
    out[:, :L, :, 0::2] = even * c - odd * s
    out[:, :L, :, 1::2] = odd * c + even * s
    return out


def swin_attention_rope(q, k, v, H, W, window, shift, pad_mode=0, theta=10000.0, scale=1.0,
                        y0=0.0, x0=0.0):
    """Flash Swin attention of RoPE-rotated q and k (v untouched): the textbook form."""
    qr = apply_rope(q, H, W, theta, scale, y0, x0)
    kr = apply_rope(k, H, W, theta, scale, y0, x0)
    return swin_attention_textbook(qr, kr, _f64(v), H, W, window, shift, pad_mode)


def swin_attention_rope_at(q, k, v, H, W, window, shift, pad_mode, queries, theta=10000.0,
                           scale=1.0):
    """RoPE attention at sampled (b, y, x) queries only (full-size checks)."""
    from .swin_oracle import swin_attention_at
    return swin_attention_at(apply_rope(q, H, W, theta, scale), apply_rope(k, H, W, theta, scale),
                             _f64(v), H, W, window, shift, pad_mode, queries)


def swin_attention_rope_lse(q, k, v, H, W, window, shift, pad_mode=0, theta=10000.0, scale=1.0):
    """Log-sum-exp of the RoPE attention: that of the rotated q and k."""
    from .backward import swin_attention_lse
    return swin_attention_lse(apply_rope(q, H, W, theta, scale), apply_rope(k, H, W, theta, scale), _f64(v),
                              H, W, window, shift, pad_mode)


def swin_attention_rope_bwd(q, k, v, dout, H, W, window, shift, pad_mode=0, theta=10000.0, scale=1.0):
    """Gradients of the RoPE attention with respect to the unrotated q, k and v.  With
    q' = R q and k' = R k per token (R a rotation), the chain rule gives dq = R^T dq' and
    dk = R^T dk', where dq', dk' are the attention gradients at q', k'; dv is unchanged and
    the unrotated pad token's gradient is dk'[L] itself."""
    from .backward import swin_attention_bwd
    dqr, dkr, dv = swin_attention_bwd(apply_rope(q, H, W, theta, scale), apply_rope(k, H, W, theta, scale),
                                      _f64(v), _f64(dout), H, W, window, shift, pad_mode)
    return (apply_rope(dqr, H, W, theta, scale, inverse=True),
            apply_rope(dkr, H, W, theta, scale, inverse=True), dv)


__all__ = ["rope_angles", "apply_rope", "swin_attention_rope", "swin_attention_rope_at",
           "swin_attention_rope_lse", "swin_attention_rope_bwd", "PAD_KVTOKEN"]

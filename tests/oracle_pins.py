"""Pins of the fp64 oracle: checks against facts that do not come from the oracle itself.

Each ``pin_*`` function takes the oracle module (so the mutation tests can hand in a
patched copy) and raises AssertionError when the oracle disagrees with:

* hand-derived values of the paper's index mappings (App. A, App. B) and window sizes
  (Sec. 3.3), stored under tests/golden/;
* closed forms of Eq. 1 (q = k = 0 gives region centroids; constant v gives v);
* special cases that reduce to a library routine (PyTorch's scaled_dot_product_attention
  in float64): window >= grid with no shift is global attention; no shift with a grid
  divisible by the window is reshape-partition window attention; KV-token mode with a
  zero pad token is window attention over a zero-filled canvas;
* the roll invariant: shifted windows that do not wrap equal unshifted window attention
  on the input rolled by -s, rolled back by +s;
* brute force over every query straight from the region definition.
"""
from __future__ import annotations

import math
import os

import numpy as np
import torch
import torch.nn.functional as F

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rand(rng, B, L, heads, d, extra=0):
    return (rng.standard_normal((B, L, heads, d)),
            rng.standard_normal((B, L + extra, heads, d)),
            rng.standard_normal((B, L + extra, heads, d)))


def _sdpa(q, k, v):
    """Library attention in float64: q [..., n, d], k/v [..., m, d] numpy."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    return F.scaled_dot_product_attention(t(q), t(k), t(v)).numpy()


def _wmsa(x_q, x_k, x_v, H, W, k):
    """Plain non-shifted window attention on a grid divisible by k, via the library
    routine.  Inputs [B, L, heads, d]; output [B, L, heads, d]."""
    B, L, heads, d = x_q.shape

    def part(x):
        x = x.reshape(B, H // k, k, W // k, k, heads, d).transpose(0, 1, 3, 5, 2, 4, 6)
        return x.reshape(B, -1, heads, k * k, d)

    o = _sdpa(part(x_q), part(x_k), part(x_v))
    o = o.reshape(B, H // k, W // k, heads, k, k, d).transpose(0, 1, 4, 2, 5, 3, 6)
    return o.reshape(B, L, heads, d)


# ---------------------------------------------------------------------------------------
def read_index_golden():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "fla_index_mappings.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key == "case":
                cur = {kv.split("=")[0]: int(kv.split("=")[1]) for kv in vals}
                cases.append(cur)
            else:
                cur[key] = [int(x) for x in vals]
    return cases


def pin_index_golden(O):
    for c in read_index_golden():
        idx, lengths, inv = O.fla_shift_window_indices(c["h"], c["w"], c["k"], c["s"])
        kv, kvl = O.fla_kv_padding_indices(c["h"], c["w"], c["k"], c["s"])
        assert idx.tolist() == c["indices"], c
        assert lengths.tolist() == c["lengths"], c
        assert kv.tolist() == c["kv_indices"], c
        assert kvl.tolist() == c["kv_lengths"], c
        x = np.arange(c["h"] * c["w"]) * 7 + 3
        assert (x[idx][inv] == x).all()


def read_histograms():
    hist, flops = [], []
    with open(os.path.join(GOLDEN, "window_histograms.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line.startswith("grid"):
                lhs, rhs = line.split(":", 1)
                H, W, k, s = map(int, lhs.split()[1:])
                want = {int(a): int(b) for a, b in (t.split(":") for t in rhs.split())}
                hist.append((H, W, k, s, want))
            elif line.startswith("flops"):
                lhs, rhs = line.split(":")
                H, W, k, s, d, heads, B = map(int, lhs.split()[1:])
                flops.append((H, W, k, s, d, heads, B, int(rhs)))
    return hist, flops


def pin_window_histograms(O):
    hist, flops = read_histograms()
    for H, W, k, s, want in hist:
        n = O.window_sizes(H, W, k, s)
        got = {}
        for x in n.tolist():
            got[x] = got.get(x, 0) + 1
        assert got == want, (H, W, got, want)
        assert n.sum() == H * W
    for H, W, k, s, d, heads, B, want in flops:
        f, _ = O.work_counts(B, heads, H, W, d, k, s, 0, 2)
        assert f == want, (H, W, f, want)


def read_centroids():
    out, grid = [], None
    with open(os.path.join(GOLDEN, "region_centroids.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            if line.startswith("grid"):
                grid = tuple(map(int, line.split()[1:]))
                out.append((grid, []))
            else:
                y, x, cy, cx, n = line.split()
                out[-1][1].append((int(y), int(x), float(cy), float(cx), int(n)))
    return out


def pin_centroids(O, forms=("swin_attention_textbook",)):
    for (H, W, k, s), pts in read_centroids():
        L = H * W
        yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
        for pad_mode in (O.PAD_MASK, O.PAD_KVTOKEN):
            extra = 1 if pad_mode == O.PAD_KVTOKEN else 0
            q = np.zeros((1, L, 1, 4))
            kk = np.zeros((1, L + extra, 1, 4))
            v = np.zeros((1, L + extra, 1, 4))
            v[0, :L, 0, 0] = yy.ravel()
            v[0, :L, 0, 1] = xx.ravel()
            v[0, :L, 0, 2] = 1.0
            for form in forms:
                out = getattr(O, form)(q, kk, v, H, W, k, s, pad_mode)
                for y, x, cy, cx, n in pts:
                    f = n / (k * k) if pad_mode == O.PAD_KVTOKEN else 1.0
                    got = out[0, y * W + x, 0]
                    want = np.array([cy * f, cx * f, f, 0.0])
                    assert np.allclose(got, want, rtol=0, atol=1e-12), (form, pad_mode, y, x, got, want)


def pin_constant_v(O, form="swin_attention_textbook"):
    rng = np.random.default_rng(11)
    for (H, W, k, s) in [(9, 11, 4, 1), (8, 8, 4, 2)]:
        for pad_mode in (O.PAD_MASK, O.PAD_KVTOKEN):
            extra = 1 if pad_mode == O.PAD_KVTOKEN else 0
            q, kk, _ = _rand(rng, 2, H * W, 2, 5, extra)
            c = rng.standard_normal((2, 1, 2, 5))
            v = np.broadcast_to(c, (2, H * W + extra, 2, 5)).copy()
            out = getattr(O, form)(q, kk, v, H, W, k, s, pad_mode)
            assert np.allclose(out, np.broadcast_to(c, out.shape), rtol=0, atol=1e-12)


def pin_global(O, form="swin_attention_textbook"):
    """window >= grid, shift 0: one window holding every token = global attention."""
    rng = np.random.default_rng(12)
    for (H, W, k) in [(5, 7, 8), (6, 6, 6), (1, 9, 9), (3, 2, 16)]:
        q, kk, v = _rand(rng, 2, H * W, 3, 8)
        out = getattr(O, form)(q, kk, v, H, W, k, 0, O.PAD_MASK)
        ref = _sdpa(q.transpose(0, 2, 1, 3), kk.transpose(0, 2, 1, 3), v.transpose(0, 2, 1, 3))
        assert np.allclose(out, ref.transpose(0, 2, 1, 3), rtol=0, atol=1e-12)


def pin_wmsa(O, form="swin_attention_textbook"):
    """shift 0 on a grid divisible by k: plain reshape-partition window attention."""
    rng = np.random.default_rng(13)
    for (H, W, k) in [(8, 12, 4), (6, 6, 3), (4, 8, 2)]:
        for pad_mode in (O.PAD_MASK, O.PAD_KVTOKEN):
            extra = 1 if pad_mode == O.PAD_KVTOKEN else 0
            q, kk, v = _rand(rng, 2, H * W, 2, 6, extra)
            out = getattr(O, form)(q, kk, v, H, W, k, 0, pad_mode)
            ref = _wmsa(q, kk[:, :H * W], v[:, :H * W], H, W, k)
            assert np.allclose(out, ref, rtol=0, atol=1e-12)


def pin_roll_invariant(O, form="swin_attention_textbook"):
    """For a grid divisible by k: shifted-window output at queries whose window does not
    wrap round the border equals roll(+s) . W-MSA . roll(-s) of the input; at queries of
    the wrapping windows the two differ (that is what the shift mask is for)."""
    rng = np.random.default_rng(14)
    for (H, W, k, s) in [(12, 12, 4, 1), (8, 12, 4, 2), (16, 16, 8, 3)]:
        q, kk, v = _rand(rng, 1, H * W, 2, 6)
        out = getattr(O, form)(q, kk, v, H, W, k, s, O.PAD_MASK)

        def roll(x, sh):
            g = x.reshape(1, H, W, 2, 6)
            return np.roll(g, (sh, sh), axis=(1, 2)).reshape(1, H * W, 2, 6)

        ref = roll(_wmsa(roll(q, -s), roll(kk, -s), roll(v, -s), H, W, k), s)
        ys = np.arange(H)
        xs = np.arange(W)
        inner_y = (ys >= s) & (ys < H - k + s)
        inner_x = (xs >= s) & (xs < W - k + s)
        inner = (inner_y[:, None] & inner_x[None, :]).ravel()
        assert np.allclose(out[:, inner], ref[:, inner], rtol=0, atol=1e-12)
        assert not np.allclose(out[:, ~inner], ref[:, ~inner], rtol=0, atol=1e-6)


def pin_kvtoken_zero_canvas(O, form="swin_attention_textbook"):
    """KV-token mode with a zero pad token = window attention over the canvas in which the
    grid sits at offset k - s and every other slot is a zero vector (q, k and v)."""
    rng = np.random.default_rng(15)
    for (H, W, k, s) in [(8, 8, 4, 2), (7, 10, 4, 1), (5, 5, 3, 0)]:
        q, kk, v = _rand(rng, 2, H * W, 2, 5, 1)
        kk[:, -1] = 0.0
        v[:, -1] = 0.0
        out = getattr(O, form)(q, kk, v, H, W, k, s, O.PAD_KVTOKEN)
        o = (k - s) % k
        Hc = -(-(H + o) // k) * k
        Wc = -(-(W + o) // k) * k

        def canvas(x):
            c = np.zeros((2, Hc, Wc, 2, 5))
            c[:, o:o + H, o:o + W] = x[:, :H * W].reshape(2, H, W, 2, 5)
            return c.reshape(2, Hc * Wc, 2, 5)

        ref = _wmsa(canvas(q), canvas(kk), canvas(v), Hc, Wc, k)
        ref = ref.reshape(2, Hc, Wc, 2, 5)[:, o:o + H, o:o + W].reshape(2, H * W, 2, 5)
        assert np.allclose(out, ref, rtol=0, atol=1e-12)


def pin_bruteforce(O, forms=("swin_attention_textbook", "swin_attention_canvas", "swin_attention_fla")):
    """Every form against the per-query region definition on small grids."""
    rng = np.random.default_rng(16)
    shapes = [(7, 9, 4, 1), (8, 8, 4, 2), (6, 10, 3, 2), (5, 3, 8, 5), (1, 1, 1, 0), (10, 7, 5, 4)]
    for (H, W, k, s) in shapes:
        for pad_mode in (O.PAD_MASK, O.PAD_KVTOKEN):
            extra = 1 if pad_mode == O.PAD_KVTOKEN else 0
            q, kk, v = _rand(rng, 2, H * W, 2, 4, extra)
            ref = O.swin_attention_bruteforce(q, kk, v, H, W, k, s, pad_mode)
            for form in forms:
                out = getattr(O, form)(q, kk, v, H, W, k, s, pad_mode)
                assert np.allclose(out, ref, rtol=0, atol=1e-12), (form, H, W, k, s, pad_mode)


ALL_PINS = [pin_index_golden, pin_window_histograms, pin_centroids, pin_constant_v, pin_global,
            pin_wmsa, pin_roll_invariant, pin_kvtoken_zero_canvas, pin_bruteforce]

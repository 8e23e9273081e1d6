"""Plant plausible mistakes in the oracle (CPU only) and check that its pins catch each.

A mutant replaces one helper of ``oracle.swin_oracle`` for the duration of a test; the
pins of ``oracle_pins`` must then fail somewhere.  This guards against pins that would
pass whatever the oracle computed."""
import math
import types

import numpy as np
import pytest

import oracle.swin_oracle as M
import oracle_pins as P

_orig = {name: getattr(M, name) for name in dir(M) if name.startswith("_") and callable(getattr(M, name))}


def _partition_xy_swapped(x, k):
    B, Hp, Wp, heads, d = x.shape
    x = x.reshape(B, Hp // k, k, Wp // k, k, heads, d).transpose(0, 1, 3, 5, 4, 2, 6)
    return x.reshape(B, (Hp // k) * (Wp // k), heads, k * k, d)


def _labels_off_by_one(n, k, s):
    lab = np.zeros(n, dtype=np.int64)
    if s > 0:
        lab[n - k + 1: n - s] = 1
        lab[n - s:] = 2
    return lab


def _softmax_wrong_axis(logits, weights):
    with np.errstate(invalid="ignore", divide="ignore"):
        z = np.where(weights > 0, logits, -np.inf)
        e = weights * np.exp(z - z.max(axis=-1, keepdims=True))
        return e / e.sum(axis=-2, keepdims=True)


def _softmax_mask_ignored(logits, weights):
    return _orig["_softmax_weighted"](logits, np.ones_like(weights))


def _window_attention_qk_swapped(qw, kw, vw, allowed, scale, kpad=None, vpad=None):
    return _orig["_window_attention"](kw, qw, vw, allowed, scale, kpad, vpad)


def _window_attention_pv_uses_q(qw, kw, vw, allowed, scale, kpad=None, vpad=None):
    return _orig["_window_attention"](qw, kw, qw, allowed, scale, kpad, vpad)


def _canvas_origin_is_shift(H, W, k, s):
    o = s
    return o, -(-(H + o) // k) * k, -(-(W + o) // k) * k


_orig_slots = M._canvas_coords


def _slots_origin_is_shift(H, W, k, s):
    # the index-list form's canvas with s virtual tokens in front instead of k - s
    return _orig_slots(H, W, k, (k - s) % k)


def _slots_column_major(H, W, k, s):
    # slots numbered column-major inside each window
    out = _orig_slots(H, W, k, s)
    return out.reshape(-1, k, k).transpose(0, 2, 1).reshape(-1, k * k)


MUTANTS = {
    "index_list_origin_is_shift": {"_canvas_coords": _slots_origin_is_shift},
    "index_list_slots_column_major": {"_canvas_coords": _slots_column_major},
    "roll_sign_flipped": {"_cyclic_shift": lambda x, s, axes: np.roll(x, (s, s), axis=axes),
                          "_cyclic_unshift": lambda x, s, axes: np.roll(x, (-s, -s), axis=axes)},
    "shift_back_missing": {"_cyclic_unshift": lambda x, s, axes: x},
    "region_slice_off_by_one": {"_region_labels_1d": _labels_off_by_one},
    "no_region_mask": {"_region_labels_1d": lambda n, k, s: np.zeros(n, dtype=np.int64)},
    "scale_one_over_d": {"math": types.SimpleNamespace(sqrt=lambda x: x)},
    "scale_missing": {"math": types.SimpleNamespace(sqrt=lambda x: 1.0)},
    "window_order_transposed": {"_partition": _partition_xy_swapped},
    "pad_keys_not_masked": {"_partition_map": lambda m, k: _orig["_partition_map"](
        np.ones_like(m) if m.dtype == bool else m, k)},
    "pad_multiplicity_off_by_one": {"_pad_multiplicity": lambda a: a.shape[1] - a.sum(axis=1) + 1},
    "pad_counted_once": {"_pad_multiplicity": lambda a: np.minimum(a.shape[1] - a.sum(axis=1), 1)},
    "softmax_wrong_axis": {"_softmax_weighted": _softmax_wrong_axis},
    "softmax_ignores_mask": {"_softmax_weighted": _softmax_mask_ignored},
    "q_and_k_swapped": {"_window_attention": _window_attention_qk_swapped},
    "pv_multiplies_q": {"_window_attention": _window_attention_pv_uses_q},
    "canvas_offset_is_shift": {"_canvas_geometry": _canvas_origin_is_shift},
    "region_rule_sign": {"_region": lambda c, k, s: np.floor_divide(np.asarray(c) + s, k)},
    "region_rule_no_shift": {"_region": lambda c, k, s: np.floor_divide(np.asarray(c), k)},
}


def _run_pins():
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(M)
        except Exception as e:  # an assertion, or a crash the mutant caused
            failed.append((pin.__name__, type(e).__name__))
    return failed


def test_unmutated_oracle_passes_every_pin():
    assert _run_pins() == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    for attr, repl in MUTANTS[name].items():
        monkeypatch.setattr(M, attr, repl)
    failed = _run_pins()
    assert failed, "mutant %s passed every pin" % name

"""The fp64 backward oracle against its pins, and planted mistakes that the pins must catch
(CPU only)."""
import math

import numpy as np
import pytest

import backward_pins as P
import oracle.backward as M

_orig = {name: getattr(M, name) for name in ("_key_sets", "_weighted_probs", "_region_keys",
                                             "_region_grads")}


@pytest.mark.parametrize("pin", P.PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(M)


def _grads_variant(**flags):
    def fn(qs, kk, vk, w, dos, c):
        z = c * np.einsum("bihd,bjhd->bhij", qs, kk)
        P, _ = _orig["_weighted_probs"](z, np.ones_like(w) if flags.get("unweighted") else w)
        o = np.einsum("bhij,bjhd->bihd", P, vk)
        D = np.einsum("bihd,bihd->bhi", dos, o)
        if flags.get("no_D"):
            D = 0 * D
        dP = np.einsum("bihd,bjhd->bhij", dos, vk)
        dz = P * (dP - D[..., None])
        cq = 1.0 if flags.get("dq_unscaled") else c
        ck = c * c if flags.get("dk_scaled_twice") else c
        dq = cq * np.einsum("bhij,bjhd->bihd", dz, kk)
        dk = ck * np.einsum("bhij,bihd->bjhd", dz, qs)
        dv = np.einsum("bhij,bihd->bjhd", dz if flags.get("dv_uses_dz") else P, dos)
        if flags.get("dk_sign"):
            dk = -dk
        return dq, dk, dv
    return fn


def _key_sets_no_shift(H, W, window, shift):
    return _orig["_key_sets"](H, W, window, 0)


def _key_sets_shift_sign(H, W, window, shift):
    return _orig["_key_sets"](H, W, window, (window - shift) % window)


def _region_keys_pad_once(q, k, v, keys, L, window, pad_mode):
    kk, vk, w = _orig["_region_keys"](q, k, v, keys, L, window, pad_mode)
    if pad_mode:
        w = w.copy()
        w[-1] = min(w[-1], 1.0)
    return kk, vk, w


def _region_keys_pad_plus_one(q, k, v, keys, L, window, pad_mode):
    kk, vk, w = _orig["_region_keys"](q, k, v, keys, L, window, pad_mode)
    if pad_mode:
        w = w.copy()
        w[-1] += 1.0
    return kk, vk, w


def _lse_base2(z, w):
    P, l = _orig["_weighted_probs"](z, w)
    return P, l / math.log(2.0)


MUTANTS = {
    "D_term_dropped": {"_region_grads": _grads_variant(no_D=True)},
    "dq_scale_missing": {"_region_grads": _grads_variant(dq_unscaled=True)},
    "dk_scaled_twice": {"_region_grads": _grads_variant(dk_scaled_twice=True)},
    "dv_from_dz": {"_region_grads": _grads_variant(dv_uses_dz=True)},
    "dk_sign_flipped": {"_region_grads": _grads_variant(dk_sign=True)},
    "pad_weight_ignored": {"_region_grads": _grads_variant(unweighted=True)},
    "regions_without_shift": {"_key_sets": _key_sets_no_shift},
    "shift_sign_flipped": {"_key_sets": _key_sets_shift_sign},
    "pad_counted_once": {"_region_keys": _region_keys_pad_once},
    "pad_multiplicity_plus_one": {"_region_keys": _region_keys_pad_plus_one},
    "lse_in_base_2": {"_weighted_probs": _lse_base2},
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    for attr, fn in MUTANTS[name].items():
        monkeypatch.setattr(M, attr, fn)
    failed = []
    for pin in P.PINS:
        try:
            pin(M)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, "mutant %s passed every pin" % name

"""Host checks of the seeded input generator (CPU): the stress rows of the key tensor are the
ones the recipe names, for one and several batch entries, with and without the pad row."""
import dataclasses

import torch

from paper_2407_02109_amd import synth


def _stressed_rows(wl):
    """Count of real key rows (b, token, head) that differ from an unstressed draw by exactly x8."""
    base = dataclasses.replace(wl, stress_keys=0.0)
    _, k, _ = synth.make_inputs(wl)
    _, k0, _ = synth.make_inputs(base)
    k, k0 = k[:, :wl.L].float(), k0[:, :wl.L].float()
    same = (k == k0).all(dim=-1)
    scaled = (k == k0 * 8.0).all(dim=-1)                     # fp32 workloads: x8 is exact
    assert bool((same | scaled).all())
    return int((~same).sum())


def _small(B, pad_mode):
    return synth.Workload("t", B, 3, 12, 10, 64, 4, 2, "f32", seed=11, stress_keys=0.05, pad_mode=pad_mode)


def test_stress_rows_counted_for_every_batch_size_and_mode():
    for B in (1, 2, 3):
        for pm in (synth.PAD_MASK, synth.PAD_KVTOKEN):
            wl = _small(B, pm)
            assert _stressed_rows(wl) == round(0.05 * B * wl.L * wl.heads), (B, pm)


def test_stress_rows_follow_the_flat_row_order():
    """In MASK mode k is contiguous, so the chosen rows are those of a flat [B*L*heads, d] view of
    k indexed by the permutation; the generator must pick exactly those (the bytes of the
    recorded workloads stay the same)."""
    for B in (1, 3):
        wl = _small(B, synth.PAD_MASK)
        _, k, _ = synth.make_inputs(wl)
        g = torch.Generator(device="cpu")
        g.manual_seed(wl.seed)
        shape = (wl.B, wl.L, wl.heads, wl.head_dim)
        torch.randn(*shape, generator=g)
        kf = torch.randn(*shape, generator=g)
        torch.randn(*shape, generator=g)
        n_rows = wl.B * wl.L * wl.heads
        hot = torch.randperm(n_rows, generator=g)[: round(wl.stress_keys * n_rows)]
        kf.view(n_rows, wl.head_dim)[hot] *= 8.0
        assert torch.equal(k, kf)
    wl = synth.WORKLOADS["img4096"]
    assert round(wl.stress_keys * wl.B * wl.L * wl.heads) == 7864

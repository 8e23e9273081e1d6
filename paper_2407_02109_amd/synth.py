"""Seeded synthetic inputs for Flash Swin attention and for Cycle-scan.

This module draws random numbers and nothing else: it holds none of the attention
arithmetic, so both the GPU tests and the fp64 oracle can consume its output.

Workloads are token grids shaped like the paper's ViT-B encoder inputs (16x16 patches,
12 heads of 64 channels, window 16, shift 8; Sec. 3.3, Sec. 4.1 and App. D): 1024^2,
2048^2 and 4096^2 images give 64x64, 128x128 and 256x256 token grids.  Values are
i.i.d. N(0, 1) from a seeded CPU generator, scaled by exact powers of two and rounded
to the storage dtype (round-to-nearest-even), so the oracle sees exactly the values the
GPU sees.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import torch

PAD_MASK = 0
PAD_KVTOKEN = 1


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    heads: int
    H: int
    W: int
    head_dim: int
    window: int
    shift: int
    dtype: str                 # "bf16" | "f32"
    seed: int
    pad_mode: int = PAD_MASK
    scale: float = 1.0         # exact power of two applied to q, k and v before rounding
    stress_keys: float = 0.0   # fraction of (token, head) key rows multiplied by 8
    grids: tuple = ()          # multi-scale: ((H, W), ...) one after the other; () = (H, W) alone
    rope: tuple = ()           # (theta, scale): 2-D RoPE on q and k inside the kernel; () = none
    note: str = field(default="", compare=False)

    @property
    def grid_list(self) -> tuple:
        return self.grids if self.grids else ((self.H, self.W),)

    @property
    def L(self) -> int:
        return sum(h * w for h, w in self.grid_list)

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny_s0": Workload("tiny_s0", 1, 1, 32, 32, 64, 8, 0, "f32", seed=0,
                        note="32x32 grid, window 8, no shift, fp32"),
    "tiny_s4": Workload("tiny_s4", 1, 1, 32, 32, 64, 8, 4, "f32", seed=0,
                        note="32x32 grid, window 8, shift 4, fp32"),
    "img1024": Workload("img1024", 1, 12, 64, 64, 64, 16, 8, "bf16", seed=1, scale=0.125,
                        note="1024^2 image: 64x64 tokens, 12 heads x 64, window 16, shift 8"),
    "img2048": Workload("img2048", 1, 12, 128, 128, 64, 16, 8, "bf16", seed=2,
                        note="2048^2 image: 128x128 tokens, 12 heads x 64, window 16, shift 8"),
    "img4096": Workload("img4096", 1, 12, 256, 256, 64, 16, 8, "bf16", seed=3, stress_keys=0.01,
                        note="4096^2 image: 256x256 tokens, 12 heads x 64, window 16, shift 8, "
                             "1% of key rows x8"),
    "img4096_kv": Workload("img4096_kv", 1, 12, 256, 256, 64, 16, 8, "bf16", seed=3, stress_keys=0.01,
                           pad_mode=PAD_KVTOKEN,
                           note="img4096 with KV-only padding: border windows attend the pad token "
                                "(row L of k and v) with multiplicity window^2 - n"),
    "img4096_rope": Workload("img4096_rope", 1, 12, 256, 256, 64, 16, 8, "bf16", seed=5,
                             rope=(10000.0, 1.0),
                             note="256x256 tokens, 12 heads x 64, window 16, shift 8, N(0,1), with 2-D RoPE "
                                  "(theta 10000, grid coordinates) applied to q and k in the kernel's prologue"),
    "ms_img2048": Workload("ms_img2048", 1, 12, 128, 128, 64, 16, 8, "bf16", seed=7,
                           pad_mode=PAD_KVTOKEN, grids=((128, 128), (32, 32)),
                           note="multi-scale (HRSAM++): the 2048^2 image's 128x128 tokens followed by "
                                "the 512^2 anchor map's 32x32, one shared pad token"),
    "img1024_w32": Workload("img1024_w32", 1, 12, 64, 64, 64, 32, 16, "bf16", seed=8,
                            note="64x64 tokens, 12 heads x 64, window 32, shift 16 (windows of 256, 512 "
                                 "and 1024 tokens): the paper's speedup shape at the wider window"),
    "img1024_w64": Workload("img1024_w64", 1, 12, 64, 64, 64, 64, 32, "bf16", seed=9,
                            note="64x64 tokens, 12 heads x 64, window 64, shift 32 (four 32x32 windows "
                                 "of 1024 tokens): the paper's speedup shape at the widest window"),
    "img4096_w32": Workload("img4096_w32", 1, 12, 256, 256, 64, 32, 16, "bf16", seed=10,
                            note="256x256 tokens, 12 heads x 64, window 32, shift 16 (1024-token windows "
                                 "inside, 512 and 256 on the border)"),
    "ragged150x203": Workload("ragged150x203", 4, 12, 150, 203, 64, 16, 8, "bf16", seed=4,
                              note="non-divisible 150x203 grid, B=4, 12 heads x 64, window 16, "
                                   "shift 8, padded keys masked"),
}


def make_inputs(wl: Workload, device: str | torch.device = "cpu"):
    """Return (q, k, v) as contiguous [B, L(+1), heads, head_dim] tensors of wl's dtype.

    In KV-token mode k and v carry one extra row (index L), the pad token, drawn like the
    others.  Generation always happens on the CPU generator so every device sees the same
    bytes."""
    g = torch.Generator(device="cpu")
    g.manual_seed(wl.seed)
    rows_kv = wl.L + (1 if wl.pad_mode == PAD_KVTOKEN else 0)
    q = torch.randn(wl.B, wl.L, wl.heads, wl.head_dim, generator=g, dtype=torch.float32)
    k = torch.randn(wl.B, rows_kv, wl.heads, wl.head_dim, generator=g, dtype=torch.float32)
    v = torch.randn(wl.B, rows_kv, wl.heads, wl.head_dim, generator=g, dtype=torch.float32)
    if wl.scale != 1.0:
        q.mul_(wl.scale)
        k.mul_(wl.scale)
        v.mul_(wl.scale)
    if wl.stress_keys > 0:
        n_rows = wl.B * wl.L * wl.heads
        n_hot = int(round(wl.stress_keys * n_rows))
        hot = torch.randperm(n_rows, generator=g)[:n_hot]
        # hot indexes the real key rows in (b, token, head) order; scaled in place through
        # explicit indices, since k[:, :L] is not contiguous when k carries a pad row
        b, rem = hot // (wl.L * wl.heads), hot % (wl.L * wl.heads)
        k[b, rem // wl.heads, rem % wl.heads] *= 8.0
    dt = wl.torch_dtype
    out = []
    for t in (q, k, v):
        t = t.to(dt).contiguous()
        out.append(t.to(device) if str(device) != "cpu" else t)
    return tuple(out)


def make_grad(wl: Workload, device: str | torch.device = "cpu"):
    """Upstream gradient dOut for a backward pass: N(0, 1) of q's shape, drawn from its own
    generator seeded with wl.seed + 1000 (so q, k, v stay those of make_inputs), rounded to
    wl's dtype."""
    g = torch.Generator(device="cpu")
    g.manual_seed(wl.seed + 1000)
    t = torch.randn(wl.B, wl.L, wl.heads, wl.head_dim, generator=g, dtype=torch.float32)
    t = t.to(wl.torch_dtype).contiguous()
    return t.to(device) if str(device) != "cpu" else t


def to_f64_numpy(t):
    """Exact float64 copy of a CPU/GPU tensor (bf16 and fp32 embed exactly in fp64)."""
    return t.detach().to("cpu", torch.float64).numpy()


def random_ms_queries(wl: Workload, n: int, seed: int):
    """n random (b, grid, y, x) query positions over the grids of a multi-scale workload, in
    proportion to their token counts, plus the four corners of every grid; int64 [S, 4]."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    grids = wl.grid_list
    sizes = torch.tensor([h * w for h, w in grids], dtype=torch.float64)
    gi = torch.multinomial(sizes / sizes.sum(), n, replacement=True, generator=g)
    b = torch.randint(0, wl.B, (n,), generator=g)
    u = torch.rand(n, 2, generator=g, dtype=torch.float64)
    hs = torch.tensor([h for h, _ in grids])[gi]
    ws = torch.tensor([w for _, w in grids])[gi]
    y = (u[:, 0] * hs).long().clamp(max=hs - 1)
    x = (u[:, 1] * ws).long().clamp(max=ws - 1)
    pts = [torch.stack([b, gi, y, x], dim=1)]
    corners = [(0, i, yy, xx) for i, (h, w) in enumerate(grids) for yy in {0, h - 1} for xx in {0, w - 1}]
    pts.append(torch.tensor(corners, dtype=torch.int64))
    return torch.cat(pts, dim=0)


def random_queries(wl: Workload, n: int, seed: int):
    """n random (b, y, x) query positions, plus every corner of the grid (the windows
    that the shift splits), as an int64 tensor [S, 3]."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    b = torch.randint(0, wl.B, (n,), generator=g)
    y = torch.randint(0, wl.H, (n,), generator=g)
    x = torch.randint(0, wl.W, (n,), generator=g)
    pts = [torch.stack([b, y, x], dim=1)]
    corners = []
    for bb in {0, wl.B - 1}:
        for yy in {0, wl.H - 1}:
            for xx in {0, wl.W - 1}:
                corners.append((bb, yy, xx))
    pts.append(torch.tensor(corners, dtype=torch.int64))
    return torch.cat(pts, dim=0)


# ---- Cycle-scan (Sec. 3.5) ----------------------------------------------------------------

@dataclass(frozen=True)
class CycleWorkload:
    name: str
    B: int
    L: int          # tokens
    d: int          # channels
    N: int          # states per channel
    repeats: int    # copies of the sequence (3 in the paper)
    seed: int
    kind: str = "mamba"
    note: str = field(default="", compare=False)


CYCLE_WORKLOADS = {
    "cyclescan_img4096": CycleWorkload(
        "cyclescan_img4096", 1, 256 * 256, 768, 32, 3, 21,
        note="4096^2 image: 256x256 tokens of the ViT-B width 768, 32 states (Sec. 3.5, App. D), three copies"),
    "cyclescan_img1024": CycleWorkload(
        "cyclescan_img1024", 1, 64 * 64, 768, 32, 3, 22, note="1024^2 image: 64x64 tokens"),
}


def make_cycle_inputs(B, L, d, N, seed, kind="mamba", device="cpu"):
    """(x, delta, A, Bm, Cm) as fp32 tensors: x, delta [B, L, d]; A [d, N]; Bm, Cm [B, L, N].
    kind "mamba" follows Mamba's initialisation: step sizes log-uniform in [0.001, 0.1],
    A = -(1, 2, ..., N) for every channel (the real S4D start), x, B, C i.i.d. N(0, 1).
    kind "wide": step sizes exp(N(-1.5, 0.5)), A uniform in [-3, -0.25] per entry."""
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(B, L, d, generator=g)
    Bm = torch.randn(B, L, N, generator=g)
    Cm = torch.randn(B, L, N, generator=g)
    if kind == "mamba":
        u = torch.rand(B, L, d, generator=g)
        delta = torch.exp(torch.log(torch.tensor(1e-3)) + u * (torch.log(torch.tensor(1e-1)) - torch.log(torch.tensor(1e-3))))
        A = -torch.arange(1, N + 1, dtype=torch.float32).repeat(d, 1)
    elif kind == "wide":
        delta = torch.exp(-1.5 + 0.5 * torch.randn(B, L, d, generator=g))
        A = -(0.25 + 2.75 * torch.rand(d, N, generator=g))
    else:
        raise ValueError(kind)
    return tuple(t.to(torch.float32).contiguous().to(device) for t in (x, delta, A, Bm, Cm))


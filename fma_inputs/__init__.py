"""Seeded synthetic workloads for the FMA forward pass.

This module only draws random inputs; it contains none of the method's
arithmetic.  Both the GPU path's tests/benchmark and the CPU oracle take their
inputs from here, so the two sides always see the same values.

The five workloads mirror the shapes of the paper's experiments (Sec. 4): a
12-head, head-dim-64 decoder for autoregressive language modelling
(enwik8-like, causal), a bidirectional masked-LM encoder (WikiText-103-like)
at long context, and a 2D vision map (a 512x512 crop at stride 4 gives a
128x128 token grid, ADE20K-like).  No dataset item is used: queries, keys and
values are i.i.d. standard normal draws standing in for projected activations,
and the learned down-sampling weights are i.i.d. N(0, 1/kernel_len) draws
standing in for trained ones.

Draw order for a workload with seed s (one torch generator, CPU for the parity tests):
  Q, K, V          randn [B, H, n, d] float32 (times qkv_scale)
  for l = 1 .. L-1, for basis b = 0 .. rank-1:
                   pi^k_{l,b} then pi^v_{l,b}, each randn [H, s_l] / sqrt(s_l)   (1D)
                   pi^{k,x}_{l,b}, pi^{k,y}_{l,b}, pi^{v,x}_{l,b}, pi^{v,y}_{l,b}
                   each randn [H, s_l] / sqrt(s_l)                               (2D)
(rank 1 is the single-vector form; the paper's experiments use rank 4)
bf16 workloads then round Q, K, V to bfloat16 (round to nearest even); the
weights stay float32.
"""
from __future__ import annotations

import dataclasses
import math

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    ndim: int            # 1 or 2
    causal: bool
    dtype: str           # "f32" or "bf16"
    batch: int
    heads: int
    n: int               # tokens (2D: rows * side)
    head_dim: int
    block: int           # base cell size r (1D block length, 2D cell side)
    side: int = 0        # 2D grid width W
    qkv_scale: float = 1.0
    seed: int = 0
    note: str = ""
    rank: int = 1        # basis vectors per level
    height: int = 0      # 2D grid height H (rows); 0: a square grid (H = W)

    @property
    def rows(self):
        """2D: the grid's rows (H)."""
        return self.height or self.side

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def _levels(ratio: int) -> int:
    # depth of the hierarchy, needed here only to know how many weight
    # vectors to draw
    L, p = 0, 1
    while p < ratio:
        p, L = 2 * p, L + 1
    return L


def level_sizes(w: Workload) -> list[int]:
    """Lengths s_l = r * 2^(l-1) of the weight vectors, l = 1 .. L-1."""
    ratio = (max(w.rows, w.side) if w.ndim == 2 else w.n) // w.block
    return [w.block * 2 ** (l - 1) for l in range(1, _levels(ratio))]


WORKLOADS = {
    "C1": Workload("C1", 1, False, "f32", 1, 1, 1024, 64, 64, seed=1961,
                   note="1D bidirectional, fp32, small case"),
    "C2": Workload("C2", 1, True, "bf16", 4, 8, 4096, 64, 64, seed=1962,
                   note="1D causal, bf16"),
    "C3": Workload("C3", 1, True, "bf16", 8, 12, 16384, 64, 128,
                   qkv_scale=1.0 / math.sqrt(64), seed=1963,
                   note="1D causal autoregressive-LM shape, bf16"),
    "C4": Workload("C4", 1, False, "bf16", 2, 16, 65536, 64, 128, seed=1964,
                   note="1D bidirectional long-context masked-LM shape, bf16"),
    "C5": Workload("C5", 2, False, "bf16", 16, 8, 128 * 128, 64, 8, side=128, seed=1965,
                   note="2D vision shape, 128x128 token grid, bf16"),
}


def custom(name="custom", ndim=1, causal=False, dtype="bf16", batch=1, heads=1, n=1024,
           head_dim=64, block=64, side=0, qkv_scale=1.0, seed=0, rank=1, height=0) -> Workload:
    """2D: a grid of `height` rows (0: square) by `side` columns."""
    if ndim == 2 and side == 0:
        side = int(round(math.sqrt(n)))
    if ndim == 2:
        n = (height or side) * side
    return Workload(name, ndim, causal, dtype, batch, heads, n, head_dim, block, side,
                    qkv_scale, seed, rank=rank, height=height if height != side else 0)


def with_rank(w: Workload, rank: int) -> Workload:
    """The same workload with `rank` basis vectors per level."""
    return dataclasses.replace(w, name="%s_p%d" % (w.name, rank), rank=rank)


def make_inputs(w: Workload, seed: int | None = None, weights_shared: bool = False,
                device: str | torch.device = "cpu"):
    """Draw (q, k, v, wk, wv) with a generator on `device` (CPU by default;
    the same seed on another device gives different, equally distributed
    values).

    q, k, v: [B, H, n, d] in the workload dtype.
    wk, wv : float32 [H, wlen] (or [wlen] when weights_shared), the level
             vectors concatenated in ascending level order, per level its
             `rank` basis vectors one after the other (2D: per basis the x
             vector then the y vector).
    """
    g = torch.Generator(device=device)
    g.manual_seed(w.seed if seed is None else seed)
    shape = (w.batch, w.heads, w.n, w.head_dim)
    dt = w.torch_dtype
    # draw in fp32, round each tensor to the workload dtype as soon as it is drawn
    q = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    if w.qkv_scale != 1.0:
        q.mul_(w.qkv_scale)
    q = q.to(dt)
    k = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    if w.qkv_scale != 1.0:
        k.mul_(w.qkv_scale)
    k = k.to(dt)
    v = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    if w.qkv_scale != 1.0:
        v.mul_(w.qkv_scale)
    v = v.to(dt)
    hw = 1 if weights_shared else w.heads
    pk, pv = [], []
    for s in [s for s in level_sizes(w) for _ in range(w.rank)]:
        if w.ndim == 1:
            pk.append(torch.randn((hw, s), generator=g, device=device) / math.sqrt(s))
            pv.append(torch.randn((hw, s), generator=g, device=device) / math.sqrt(s))
        else:
            kx = torch.randn((hw, s), generator=g, device=device) / math.sqrt(s)
            ky = torch.randn((hw, s), generator=g, device=device) / math.sqrt(s)
            vx = torch.randn((hw, s), generator=g, device=device) / math.sqrt(s)
            vy = torch.randn((hw, s), generator=g, device=device) / math.sqrt(s)
            pk += [kx, ky]
            pv += [vx, vy]
    if pk:
        wk = torch.cat(pk, dim=1).contiguous()
        wv = torch.cat(pv, dim=1).contiguous()
    else:
        wk = torch.zeros((hw, 0), device=device)
        wv = torch.zeros((hw, 0), device=device)
    if weights_shared:
        wk, wv = wk[0].contiguous(), wv[0].contiguous()
    return q, k, v, wk, wv


def make_query_weights(w: Workload, weights_shared: bool = False, device: str | torch.device = "cpu"):
    """FMA-linear query aggregation weights pi^q, laid out like pi^k ([H, wlen]
    or [wlen]), i.i.d. N(0, 1/s_l) like the others, from their own generator
    (seed + 1) so that the other inputs do not change."""
    g = torch.Generator(device=device)
    g.manual_seed(w.seed + 1)
    hw = 1 if weights_shared else w.heads
    parts = []
    for s in [s for s in level_sizes(w) for _ in range(w.rank)]:
        for _ in range(1 if w.ndim == 1 else 2):
            parts.append(torch.randn((hw, s), generator=g, device=device) / math.sqrt(s))
    wq = torch.cat(parts, dim=1).contiguous() if parts else torch.zeros((hw, 0), device=device)
    return wq[0].contiguous() if weights_shared else wq


# softmax scale whose product with log2(e) is exactly 1 in float32: scores
# in base-2 units then equal the plain dot products
PEAKED_SCALE = 0.6931471824645996   # float32(ln 2)


def make_peaked_inputs(w: Workload, seed: int | None = None, device: str | torch.device = "cpu"):
    """Inputs on which every softmax row is sharply peaked and every score is
    exact in bf16 / fp32 arithmetic, for structural checks of masks and lists.

    q, k   : integers drawn uniformly from [-2, 2] (exact in bf16), so that
             q . k is an exact integer with a spread of ~16; with
             softmax_scale = PEAKED_SCALE those are the base-2 scores, and one
             source dominates each row by several units;
    v      : standard normal, rounded to the workload dtype;
    wk, wv : every weight vector one-hot at an offset drawn per head, level
             and basis (2D: per axis), so that an aggregated key or value is
             exactly one token of its group.
    Shapes and layouts as make_inputs (per-head weights)."""
    g = torch.Generator(device=device)
    g.manual_seed(w.seed if seed is None else seed)
    shape = (w.batch, w.heads, w.n, w.head_dim)
    dt = w.torch_dtype
    q = torch.randint(-2, 3, shape, generator=g, device=device).to(dt)
    k = torch.randint(-2, 3, shape, generator=g, device=device).to(dt)
    v = torch.randn(shape, generator=g, dtype=torch.float32, device=device).to(dt)
    pk, pv = [], []

    def onehot(s):
        x = torch.zeros((w.heads, s), device=device)
        idx = torch.randint(0, s, (w.heads,), generator=g, device=device)
        x[torch.arange(w.heads, device=device), idx] = 1.0
        return x

    for s in [s for s in level_sizes(w) for _ in range(w.rank)]:
        for _ in range(1 if w.ndim == 1 else 2):
            pk.append(onehot(s))
        for _ in range(1 if w.ndim == 1 else 2):
            pv.append(onehot(s))
    if pk:
        wk = torch.cat(pk, dim=1).contiguous()
        wv = torch.cat(pv, dim=1).contiguous()
    else:
        wk = torch.zeros((w.heads, 0), device=device)
        wv = torch.zeros((w.heads, 0), device=device)
    return q, k, v, wk, wv

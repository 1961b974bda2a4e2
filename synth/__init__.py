"""Seeded synthetic inputs shaped like the global-attention layers of a VGGT-style
3D vision transformer.

This module only draws inputs. It performs none of the selection or attention
arithmetic, and both the CPU oracle and the GPU path consume exactly the arrays it
returns (bf16 tensors stored as uint16 bit patterns, float32 Gram matrices, int32
budgets).

Token layout (the sink rule of the paper's block grid, Supp. F): every view's patch
tokens, view-major, followed by all special (camera + register) tokens of every
view, so the special tokens sit in the trailing key blocks.

Recipe per head h (all draws from one numpy PCG64 stream, in this order):
  F_h, G_h  in R^{8x64}, entries N(0, 1/8)          (shared low-rank factors)
  c_h       in R^8,  N(0, I)                          (scene code)
  a_v       = c_h + N(0, I)      for each view v      (view codes)
  then for X in (Q, K, V):
    z_t     = a_{view(t)} + N(0, I)   for patch tokens, view-major
    z_t     = 2 c_h + 0.1 N(0, I)     for special tokens (sinks)
    eps     = N(0, 1) in R^{N x 64}
    Q = 0.5 z F + sigma eps,  K = 0.5 z F + sigma eps,  V = 0.25 z G + sigma eps
Values are generated in float32 and rounded to bf16 (round to nearest even).

The output projection slice of head h is W_O^h = U_h diag(10^{-k/63}) R_h
(k = 0..63) with U_h in R^{1024x64} orthonormal and R_h orthogonal, drawn from a
second stream (seed + 2), so that the singular values span two decades. Because
U_h has orthonormal columns, its Gram matrix equals R_h^T diag(10^{-2k/63}) R_h,
which is how the generator writes the float32 Gram input (formed in float64,
rounded once).

Per-head keep budgets come from a target block sparsity s_h:
  c_h = floor((1 - s_h) n_kb + 1/2) - |F|,
clamped to [min(|P|, max(0, 2 - |F|)), |P|], where F is the set of key blocks that
hold special tokens and P the remaining candidate blocks (the paper's two-block
floor, Supp. F; budget-only sparsity control, Sec. 4.4).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

RANK = 8
D_MODEL = 1024
PATCH_518 = 37 * 37  # 518x518 input with 14-pixel patches
SPECIAL_PER_VIEW = 5  # 1 camera + 4 register tokens


@dataclasses.dataclass
class Layer:
    """One synthetic global-attention layer."""

    H: int
    N: int
    D: int
    bq: int
    bk: int
    n_special_tail: int
    q: np.ndarray  # uint16 [H][N][D], bf16 bit patterns
    k: np.ndarray
    v: np.ndarray
    gram: np.ndarray  # float32 [H][D][D]
    budgets: np.ndarray  # int32 [H]
    sparsity: np.ndarray  # float64 [H], the targets the budgets came from
    seed: int
    name: str = ""

    @property
    def n_qb(self) -> int:
        return (self.N + self.bq - 1) // self.bq

    @property
    def n_kb(self) -> int:
        return (self.N + self.bk - 1) // self.bk

    def w_o(self) -> np.ndarray:
        """float64 [H][1024][D]: the output-projection slices behind `gram`."""
        return draw_w_o(self.H, self.D, self.seed)[0]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def forced_block_count(N: int, bk: int, n_special_tail: int) -> int:
    """Number of trailing key blocks that overlap the special-token tail."""
    if n_special_tail <= 0 or N == 0:
        return 0
    n_kb = (N + bk - 1) // bk
    first = (N - n_special_tail) // bk
    return n_kb - first


def budgets_from_sparsity(sparsity, N: int, bk: int, n_special_tail: int) -> np.ndarray:
    n_kb = (N + bk - 1) // bk
    nf = forced_block_count(N, bk, n_special_tail)
    n_p = n_kb - nf
    lo = min(n_p, max(0, 2 - nf))
    out = []
    for s in np.atleast_1d(sparsity):
        c = int(math.floor((1.0 - float(s)) * n_kb + 0.5)) - nf
        out.append(min(max(c, lo), n_p))
    return np.asarray(out, dtype=np.int32)


def draw_w_o(H: int, D: int, seed: int):
    """Output-projection slices W_O^h = U diag(sig) R and their float32 Gram matrices."""
    rng = np.random.default_rng(seed + 2)
    sig = 10.0 ** (-np.arange(D) / (D - 1))
    w = np.empty((H, D_MODEL, D), dtype=np.float64)
    gram = np.empty((H, D, D), dtype=np.float32)
    for h in range(H):
        u, _ = np.linalg.qr(rng.standard_normal((D_MODEL, D)))
        r, rr = np.linalg.qr(rng.standard_normal((D, D)))
        r = r * np.sign(np.diag(rr))[None, :]
        w[h] = (u * sig[None, :]) @ r
        gram[h] = ((r.T * (sig ** 2)[None, :]) @ r).astype(np.float32)
    return w, gram


def make_layer(views: int, patch_per_view: int, special_per_view: int, *, H: int = 16,
               D: int = 64, block: int = 128, sigma: float = 0.5, sparsity=0.75,
               seed: int = 1000, name: str = "", bq: int | None = None,
               bk: int | None = None) -> Layer:
    """Draw one layer: `views` views of `patch_per_view` patch tokens plus
    `special_per_view` special tokens each (all special tokens trail)."""
    bq = block if bq is None else bq
    bk = block if bk is None else bk
    n_patch = views * patch_per_view
    n_spec = views * special_per_view
    N = n_patch + n_spec
    rng = np.random.default_rng(seed)
    q = np.empty((H, N, D), dtype=np.uint16)
    k = np.empty_like(q)
    v = np.empty_like(q)
    view_of = np.repeat(np.arange(views), patch_per_view)
    f32 = np.float32
    for h in range(H):
        F = rng.standard_normal((RANK, D), dtype=f32) * f32(math.sqrt(1.0 / RANK))
        G = rng.standard_normal((RANK, D), dtype=f32) * f32(math.sqrt(1.0 / RANK))
        c = rng.standard_normal(RANK, dtype=f32)
        a = c[None, :] + rng.standard_normal((views, RANK), dtype=f32)
        for out, fac, amp in ((q, F, 0.5), (k, F, 0.5), (v, G, 0.25)):
            z = np.empty((N, RANK), dtype=f32)
            z[:n_patch] = a[view_of] + rng.standard_normal((n_patch, RANK), dtype=f32)
            z[n_patch:] = 2.0 * c[None, :] + f32(0.1) * rng.standard_normal((n_spec, RANK), dtype=f32)
            x = f32(amp) * (z @ fac)
            x += f32(sigma) * rng.standard_normal((N, D), dtype=f32)
            out[h] = f32_to_bf16_bits(x)
    _, gram = draw_w_o(H, D, seed)
    sp = np.broadcast_to(np.asarray(sparsity, dtype=np.float64), (H,)).copy()
    budgets = budgets_from_sparsity(sp, N, bk, n_spec)
    return Layer(H=H, N=N, D=D, bq=bq, bk=bk, n_special_tail=n_spec, q=q, k=k, v=v,
                 gram=gram, budgets=budgets, sparsity=sp, seed=seed, name=name)


# The five workloads: (views, patch tokens/view, special tokens/view, block, sparsity,
# restoration rounds). Seeds are 1000 + workload index (+ layer index for the stack).
CONFIGS = {
    "tiny": dict(index=0, views=4, patch=256, special=0, block=64, sparsity=(0.5,), rounds=(3,)),
    "8v": dict(index=1, views=8, patch=PATCH_518, special=SPECIAL_PER_VIEW, block=128,
               sparsity=(0.5, 0.75), rounds=(5,)),
    "32v": dict(index=2, views=32, patch=PATCH_518, special=SPECIAL_PER_VIEW, block=128,
                sparsity=(0.75, 0.9), rounds=(1, 3, 5)),
    "100v": dict(index=3, views=100, patch=PATCH_518, special=SPECIAL_PER_VIEW, block=128,
                 sparsity=("ragged",), rounds=(5,)),
    "16v_stack": dict(index=4, views=16, patch=PATCH_518, special=SPECIAL_PER_VIEW, block=128,
                      sparsity=(0.75,), rounds=(5,), layers=24),
}


def stack_sigma(layer: int, n_layers: int = 24) -> float:
    """Noise scale of layer `layer` in the layer stack: 0.3 rising to 1.0."""
    return 0.3 + 0.7 * layer / (n_layers - 1)


def make_config(name: str, sparsity=None, layer: int = 0, H: int = 16, bq=None, bk=None) -> Layer:
    """One layer of a named workload; bq / bk override its block sizes (for
    instance the 128-query / 64-key grid)."""
    cfg = CONFIGS[name]
    seed = 1000 + cfg["index"] + (layer if name == "16v_stack" else 0)
    sigma = stack_sigma(layer) if name == "16v_stack" else 0.5
    if sparsity is None:
        sparsity = cfg["sparsity"][0]
    if isinstance(sparsity, str) and sparsity == "ragged":
        sparsity = np.random.default_rng(seed + 1).uniform(0.80, 0.95, size=H)
    return make_layer(cfg["views"], cfg["patch"], cfg["special"], H=H, block=cfg["block"],
                      sigma=sigma, sparsity=sparsity, seed=seed, name=name, bq=bq, bk=bk)

"""Direct, definition-level computations used to pin the oracle.

Nothing here retypes the oracle's formulas. Each quantity is computed from the
definition the paper starts from: the pooled map is a softmax (Eq. 1), dropping
blocks renormalises that softmax over the remaining blocks (Sec. 3, step (3);
Eqs. 3 and 11 are consequences), and the drift is measured after the output
projection (Eq. 6: ||W_O (masked output - dense output)||). The closed forms of
Eqs. 4-16 are then checked against these definitions.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
from scipy.special import softmax

import synth


def decode(u16: np.ndarray) -> np.ndarray:
    return synth.bf16_bits_to_f32(u16).astype(np.float64)


def pool_numpy(x_u16: np.ndarray, b: int) -> np.ndarray:
    """Block means via numpy's own mean (Sec. 3, step (1))."""
    x = decode(x_u16)
    H, N, D = x.shape
    nb = (N + b - 1) // b
    out = np.zeros((H, nb, D))
    for i in range(nb):
        out[:, i] = x[:, i * b:min((i + 1) * b, N)].mean(axis=1)
    return out


def pooled_logits(qbar_i: np.ndarray, kbar: np.ndarray) -> np.ndarray:
    return kbar @ qbar_i / math.sqrt(kbar.shape[1])


def masked_output(logits: np.ndarray, vbar: np.ndarray, keep: np.ndarray) -> np.ndarray:
    """Pooled attention output when only `keep` blocks remain, the softmax being
    renormalised over them."""
    z = np.where(keep, logits, -np.inf)
    return softmax(z) @ vbar


def drift_vec(logits, vbar, drop):
    """Change of the pooled attention output caused by dropping `drop`."""
    full = np.ones_like(drop, dtype=bool)
    return masked_output(logits, vbar, ~drop) - masked_output(logits, vbar, full)


def drift_sq_w(logits, vbar, W, drop) -> float:
    """||W_O (masked output - dense output)||^2 with the materialised W_O slice."""
    return float(np.sum((W @ drift_vec(logits, vbar, drop)) ** 2))


def drift_sq_m(logits, vbar, M, drop) -> float:
    """The same squared norm, measured with a Gram matrix M = W_O^T W_O."""
    dv = drift_vec(logits, vbar, drop)
    return float(dv @ M @ dv)


def top_by(values: np.ndarray, member: np.ndarray, k: int):
    """Indices of the k members with the largest value, ties to the lower index,
    plus the gap between the k-th and (k+1)-th value (inf if none)."""
    idx = np.flatnonzero(member)
    order = sorted(idx.tolist(), key=lambda j: (-values[j], j))
    chosen = np.zeros_like(member, dtype=bool)
    chosen[order[:k]] = True
    gap = values[order[k - 1]] - values[order[k]] if 0 < k < len(order) else math.inf
    return chosen, gap


def brute_force_min(logits, vbar, M, cand: np.ndarray, c: int):
    """Exact optimum of the set problem (Eq. 2) by enumerating every drop set of
    size |P| - c; returns (J*, drop mask)."""
    idx = np.flatnonzero(cand)
    best, best_set = math.inf, None
    for keep in itertools.combinations(idx.tolist(), c):
        drop = cand.copy()
        drop[list(keep)] = False
        j = drift_sq_m(logits, vbar, M, drop)
        if j < best:
            best, best_set = j, drop
    return best, best_set


def brute_force_max(logits, vbar, M, cand: np.ndarray, c: int):
    """Largest drift over every drop set of size |P| - c (the sign-flipped problem)."""
    idx = np.flatnonzero(cand)
    best = -math.inf
    for keep in itertools.combinations(idx.tolist(), c):
        drop = cand.copy()
        drop[list(keep)] = False
        best = max(best, drift_sq_m(logits, vbar, M, drop))
    return best


def row_inputs(layer, h: int, i: int, pooled=None):
    """Pooled inputs of row (h, i): qbar_i, kbar, vbar (float64), M (float64 of the
    float32 Gram), forced mask, budget, W_O slice."""
    if pooled is None:
        pooled = (pool_numpy(layer.q, layer.bq), pool_numpy(layer.k, layer.bk),
                  pool_numpy(layer.v, layer.bk))
    qb, kb, vb = pooled
    n_kb = layer.n_kb
    forced = np.zeros(n_kb, dtype=bool)
    for j in range(n_kb):
        toks = np.arange(j * layer.bk, min((j + 1) * layer.bk, layer.N))
        forced[j] = bool(np.any(toks >= layer.N - layer.n_special_tail))
    return dict(qbar_i=qb[h, i], kbar=kb[h], vbar=vb[h], M=layer.gram[h].astype(np.float64),
                forced=forced, c=int(layer.budgets[h]))

"""Single-block masking reference (Sec. 3, Fig. 2) on the library's kernels.

For each key block j, every query block attends to all key blocks except j
(ress_sparse_attn_out_f32 with the list B minus j), and the change in what
attention writes into the residual stream is measured against the unmasked
output: for query block i of head h, the Euclidean norm over its tokens t of
W_O^h (O_t(B minus j) - O_t(B)), using ||W_O^h x||^2 = x^T M_h x
(ress_block_drift_sq). Ranking the
candidate blocks of a row by this change and by a selection criterion (pooled
probability, or the drift score of Eqs. 5-7) and taking the Spearman
correlation gives the comparison of Fig. 2.
"""
from __future__ import annotations

import numpy as np
import torch

from . import ress_block_drift_sq, ress_sparse_attn_out_f32


def block_masking_change(q, k, v, gram, *, bq: int, bk: int, blocks=None, stream=None) -> np.ndarray:
    """float64 [H][n_qb][len(blocks)]: the masking change of every (head, query
    block) for each key block in `blocks` (default: every key block)."""
    H, N, D = q.shape
    n_qb, n_kb = (N + bq - 1) // bq, (N + bk - 1) // bk
    blocks = list(range(n_kb)) if blocks is None else [int(j) for j in blocks]
    dev = q.device
    every = torch.arange(n_kb, dtype=torch.int32, device=dev)
    kept_all = every.expand(H, n_qb, n_kb).contiguous()
    count_all = torch.full((H, n_qb), n_kb, dtype=torch.int32, device=dev)
    count_drop = torch.full((H, n_qb), n_kb - 1, dtype=torch.int32, device=dev)
    base = ress_sparse_attn_out_f32(q, k, v, count_all, kept_all, bq=bq, bk=bk, stream=stream)
    masked = torch.empty_like(base)
    M = gram.to(device=dev, dtype=torch.float32).contiguous()
    sq = torch.empty((H, n_qb), dtype=torch.float64, device=dev)
    out = np.empty((H, n_qb, len(blocks)))
    for col, j in enumerate(blocks):
        lst = torch.cat([every[:j], every[j + 1:], torch.full((1,), -1, dtype=torch.int32, device=dev)])
        kept = lst.expand(H, n_qb, n_kb).contiguous()
        ress_sparse_attn_out_f32(q, k, v, count_drop, kept, bq=bq, bk=bk, out=masked, stream=stream)
        ress_block_drift_sq(masked, base, M, bq=bq, out=sq, stream=stream)
        out[:, :, col] = np.sqrt(np.maximum(sq.cpu().numpy(), 0.0))
    return out


def _ranks(x: np.ndarray) -> np.ndarray:
    """Average ranks along the last axis (ties share the mean of their positions)."""
    order = np.argsort(x, axis=-1, kind="stable")
    sx = np.take_along_axis(x, order, -1)
    n = x.shape[-1]
    pos = np.broadcast_to(np.arange(n, dtype=np.float64), x.shape)
    new_run = np.concatenate([np.ones(x.shape[:-1] + (1,), bool), sx[..., 1:] != sx[..., :-1]], -1)
    run_id = np.cumsum(new_run, -1) - 1
    r_sorted = np.empty(x.shape)
    for idx in np.ndindex(x.shape[:-1]):
        ids = run_id[idx]
        sums = np.bincount(ids, weights=pos[idx])
        cnts = np.bincount(ids)
        r_sorted[idx] = (sums / cnts)[ids]
    r = np.empty(x.shape)
    np.put_along_axis(r, order, r_sorted, -1)
    return r


def spearman_rows(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Spearman correlation of a[..., :] with b[..., :] for every leading index
    (nan where a ranking is constant)."""
    ra, rb = _ranks(np.asarray(a, np.float64)), _ranks(np.asarray(b, np.float64))
    ra -= ra.mean(-1, keepdims=True)
    rb -= rb.mean(-1, keepdims=True)
    den = np.sqrt((ra * ra).sum(-1) * (rb * rb).sum(-1))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(den > 0, (ra * rb).sum(-1) / den, np.nan)

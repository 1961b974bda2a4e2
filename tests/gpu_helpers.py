"""Helpers of the GPU parity tests: run the HIP path through the C ABI on a
synthetic layer, run the oracle on the same inputs, and compare.

Tolerances (applied in compare_*):
  attention   max |O_gpu - O_ref| <= 2e-2 and mean <= 2e-3 against the float64
              oracle (bf16 inputs and outputs, bf16 MFMA products);
  keys, P, J  relative error <= 1e-3 (denominator max(|ref|, 1e-6 * row max));
              the float64 selection path is also reported against 1e-9;
  kept lists  bit-exact on every row whose oracle decision margin exceeds
              MARGIN (the smallest relative gap of any top-k cut or track-best
              comparison along the row's trajectory); on the other rows the
              GPU list must still be a valid selection, and those rows may be
              at most MAX_EXCLUDED of the compared rows (0 on the five
              workloads; the stats line reports the count).
"""
from __future__ import annotations

import functools
import math
import sys
import time

import numpy as np

import oracle
import synth

MARGIN = 1e-9
MAX_EXCLUDED = 0.01  # fraction of compared rows allowed below MARGIN
ATTN_MAX, ATTN_MEAN = 2e-2, 2e-3
REL_TOL = 1e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=24)
def stack_layer(layer: int):
    """Layer `layer` of the 24-layer stack (drawn once per test process)."""
    return synth.make_config("16v_stack", layer=layer)


def stack_w_o_bits(L):
    """The full output projection of a layer, bf16 bits [1024][1024] (out x in,
    input channel 64h + d), from the generator's per-head slices W_O^h."""
    w, _ = synth.draw_w_o(L.H, L.D, L.seed)
    return synth.f32_to_bf16_bits(w.transpose(1, 0, 2).reshape(w.shape[1], L.H * L.D).astype(np.float32))


def device_inputs(L, dev="cuda:0"):
    import torch

    import paper_2609_35593_amd as ress

    return (ress.bf16_from_bits(L.q, dev), ress.bf16_from_bits(L.k, dev), ress.bf16_from_bits(L.v, dev),
            torch.from_numpy(L.gram).to(dev))


def gpu_select(L, inputs=None, rounds=5, budgets=None, want_debug=True, dense_special_queries=True, **kw):
    import torch

    import paper_2609_35593_amd as ress

    q, k, v, gram = inputs if inputs is not None else device_inputs(L)
    b = L.budgets if budgets is None else budgets
    out = ress.ress_select(q, k, v, gram, b, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail, rounds=rounds,
                           want_debug=want_debug, dense_special_queries=dense_special_queries, **kw)
    torch.cuda.synchronize()
    return {n: (t.cpu().numpy() if t is not None else None) for n, t in out.items()}, out


def oracle_select(L, rounds=5, budgets=None, rows=None, dense_special_queries=True, criterion=0, cdf_tau=0.0):
    b = L.budgets if budgets is None else budgets
    return oracle.select(L.q, L.k, L.v, L.gram, b, N=L.N, bq=L.bq, bk=L.bk, n_special=L.n_special_tail,
                         rounds=rounds, rows=rows, dense_special_queries=dense_special_queries,
                         criterion=criterion, cdf_tau=cdf_tau)


def check_lists_valid(L, kc, ki, budgets, rows, dense_special_queries=True, capped=False):
    """Structure every kept list must have, whatever the decisions (capped: a CDF
    cap may keep fewer candidates, never fewer than two blocks in all)."""
    nf = synth.forced_block_count(L.N, L.bk, L.n_special_tail)
    forced = set(range(L.n_kb - nf, L.n_kb))
    dense_rows = dense_special_queries and L.n_special_tail > 0
    first_dense = (L.N - L.n_special_tail) // L.bq if dense_rows else L.n_qb
    for r, flat in enumerate(rows):
        h, i = divmod(int(flat), L.n_qb)
        cnt = int(kc[r])
        lst = ki[r]
        n_p = L.n_kb - nf
        expect = L.n_kb if (i >= first_dense or budgets[h] >= n_p) else int(budgets[h]) + nf
        if capped and expect < L.n_kb:
            assert min(2, L.n_kb) <= cnt <= expect, (h, i, cnt, expect)
        else:
            assert cnt == expect, (h, i, cnt, expect)
        assert np.all(np.diff(lst[:cnt]) > 0) and lst[0] >= 0 and lst[cnt - 1] < L.n_kb
        assert np.all(lst[cnt:] == -1)
        assert forced <= set(lst[:cnt].tolist())


def rel_err(a, ref, rowwise_scale):
    # The floor keeps a row whose oracle values are all zero (a single key block,
    # P = 1: e = 0 and the key is 0 by Eq. 9) at 0/1e-300 instead of 0/0; any
    # nonzero GPU value there still fails.
    den = np.maximum(np.maximum(np.abs(ref), rowwise_scale), 1e-300)
    return np.abs(a - ref) / den


def compare_select(L, gpu, ref, rows=None, budgets=None, label="", dense_special_queries=True, criterion=0,
                   capped=False, max_excluded=MAX_EXCLUDED):
    """gpu: full-layer arrays; ref: oracle outputs for `rows` (flat h*n_qb+i).
    criterion 2 / 3 maximise the drift, so the returned J is >= the initial one.
    At most `max_excluded` of the rows may fall outside the bit-exact kept-list
    comparison (oracle margin <= MARGIN); the five workloads require 0."""
    budgets = L.budgets if budgets is None else budgets
    R = L.H * L.n_qb
    rows = np.arange(R) if rows is None else np.asarray(rows)
    kc = gpu["kept_count"].reshape(R)[rows]
    ki = gpu["kept_idx"].reshape(R, L.n_kb)[rows]
    check_lists_valid(L, kc, ki, budgets, rows, dense_special_queries, capped)
    same = (kc == ref["kept_count"]) & np.all(ki == ref["kept_idx"], axis=1)
    decided = ref["margin"] > MARGIN
    bad = np.flatnonzero(decided & ~same)
    stats = dict(rows=len(rows), checked=int(decided.sum()), identical=int(same.sum()),
                 identical_frac=float(same.mean()), excluded=float(1 - decided.mean()),
                 excluded_rows=int((~decided).sum()), excluded_identical=int((~decided & same).sum()))
    assert bad.size == 0, f"{label}: {bad.size} decided rows differ, first {rows[bad[:5]]}"
    assert stats["excluded"] <= max_excluded, (
        f"{label}: {int((~decided).sum())} of {len(rows)} rows have an oracle margin <= {MARGIN} "
        f"(allowed fraction {max_excluded})")
    out = {}
    if gpu.get("key") is not None and ref.get("key") is not None:
        key_g = gpu["key"].reshape(R, L.n_kb)[rows]
        prob_g = gpu["prob"].reshape(R, L.n_kb)[rows]
        e_key = rel_err(key_g, ref["key"], 1e-6 * np.abs(ref["key"]).max(axis=1, keepdims=True))
        e_p = rel_err(prob_g, ref["prob"], 1e-6 * ref["prob"].max(axis=1, keepdims=True))
        assert e_key.max() <= REL_TOL and e_p.max() <= REL_TOL, (label, e_key.max(), e_p.max())
        out.update(key_rel_max=float(e_key.max()), prob_rel_max=float(e_p.max()))
    if gpu.get("drift") is not None:
        dr = gpu["drift"].reshape(R, 2)[rows]
        scale = 1e-6 * max(np.abs(ref["drift"]).max(), 1e-300)
        e_j0 = rel_err(dr[:, 0], ref["drift"][:, 0], scale)
        e_jb = rel_err(dr[same, 1], ref["drift"][same, 1], scale)
        assert e_j0.max() <= REL_TOL and (e_jb.size == 0 or e_jb.max() <= REL_TOL), (label, e_j0.max())
        if criterion in (2, 3):
            assert np.all(dr[:, 1] >= dr[:, 0])
        else:
            assert np.all(dr[:, 1] <= dr[:, 0])
        out.update(j_init_rel_max=float(e_j0.max()), j_best_rel_max=float(e_jb.max()) if e_jb.size else 0.0)
    stats.update(out)
    say(f"  select parity {label}: {stats}")
    return stats


def sample_tokens(L, n, seed=0):
    """Stratified query tokens: every head, the first and last query block (partial
    and special rows), plus uniform picks."""
    rng = np.random.default_rng(seed)
    hs, ts = [], []
    per_head = max(4, n // L.H)
    for h in range(L.H):
        fixed = [0, min(L.bq, L.N - 1), L.N - 1, max(0, L.N - L.n_special_tail - 1)]
        extra = rng.integers(0, L.N, size=max(0, per_head - len(fixed)))
        for t in list(fixed) + list(extra):
            hs.append(h)
            ts.append(int(t))
    return np.asarray(hs, np.int32), np.asarray(ts, np.int32)


def compare_attn(L, o_gpu, hs, ts, kept_count=None, kept_idx=None, label=""):
    import torch

    o = o_gpu[torch.from_numpy(hs.astype(np.int64)), torch.from_numpy(ts.astype(np.int64))]
    return compare_attn_values(L, o.float().cpu().numpy(), hs, ts, kept_count, kept_idx, label)


def compare_attn_values(L, o, hs, ts, kept_count=None, kept_idx=None, label=""):
    """o: the GPU outputs of the (head, token) pairs hs, ts, as float [n][D]."""
    o = np.asarray(o, np.float64)
    t0 = time.time()
    ref = oracle.attn_tokens(L.q, L.k, L.v, N=L.N, bq=L.bq, bk=L.bk, scale=1.0 / math.sqrt(L.D), sel_h=hs,
                             sel_t=ts, kept_count=kept_count, kept_idx=kept_idx)
    err = np.abs(o - ref)
    say(f"  attn parity {label}: {len(hs)} tokens, max {err.max():.3e}, mean {err.mean():.3e}, "
        f"mean|ref| {np.abs(ref).mean():.3f} (oracle {time.time() - t0:.1f}s)")
    assert np.all(np.isfinite(o)), (label, "non-finite outputs")
    assert err.max() <= ATTN_MAX and err.mean() <= ATTN_MEAN, (label, err.max(), err.mean())
    return float(err.max()), float(err.mean())

"""Seeded random small layers against the oracle: every selection row and sparse and
dense attention on every token, over random shapes (1-3 views of up to 900 patch
tokens and 0-20 special tokens each, 1-3 heads, every block grid), per-head
sparsities, round counts, selection criteria (drift, probability with and without
a CDF cap, the two drift-maximising variants) and the special-query-row flag.
The cases are drawn once from a fixed seed, so every run checks the same layers;
each case prints its parameters before it touches the GPU."""
import numpy as np
import pytest

import synth
from gpu_helpers import compare_attn, compare_select, device_inputs, gpu_select, oracle_select, say

pytestmark = pytest.mark.gpu

N_CASES = 100


def draw_cases(n=N_CASES, seed=2609):
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        views = int(rng.integers(1, 4))
        patch = int(rng.integers(0, 901))
        special = int(rng.choice([0, 0, 1, 5, 20]))
        if views * (patch + special) == 0:
            continue
        H = int(rng.integers(1, 4))
        bq, bk = (int(x) for x in rng.choice([64, 128], size=2))
        sparsity = [round(float(x), 3) for x in rng.uniform(0.1, 0.95, size=H)]
        rounds = int(rng.choice([0, 1, 2, 3, 5, 8]))
        criterion = int(rng.choice([0, 0, 0, 1, 2, 3]))
        tau = float(rng.choice([0.0, 0.8])) if criterion == 1 else 0.0
        dense_special = bool(rng.choice([True, True, False]))
        cases.append(dict(views=views, patch=patch, special=special, H=H, bq=bq, bk=bk, sparsity=sparsity,
                          rounds=rounds, criterion=criterion, tau=tau, dense_special=dense_special,
                          seed=int(rng.integers(0, 1 << 30))))
    return cases


CASES = draw_cases()


@pytest.fixture(scope="module")
def ress():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_35593_amd as r

    return r


@pytest.mark.parametrize("idx", range(N_CASES))
def test_random_small_layer(ress, idx):
    import torch

    c = CASES[idx]
    L = synth.make_layer(c["views"], c["patch"], c["special"], H=c["H"], bq=c["bq"], bk=c["bk"],
                         sparsity=np.asarray(c["sparsity"]), seed=c["seed"], name=f"random{idx}")
    label = (f"case {idx}: N={L.N} H={L.H} {L.bq}/{L.bk} special={L.n_special_tail} budgets={L.budgets.tolist()} "
             f"R={c['rounds']} criterion={c['criterion']} tau={c['tau']} dense_special={c['dense_special']}")
    say(f"[random layer] {label}")
    inputs = device_inputs(L)
    kw = dict(rounds=c["rounds"], dense_special_queries=c["dense_special"])
    gpu, dev = gpu_select(L, inputs, criterion=c["criterion"], cdf_tau=c["tau"], **kw)
    ref = oracle_select(L, criterion=c["criterion"], cdf_tau=c["tau"], **kw)
    rows = L.H * L.n_qb
    # A tiny layer has few rows: at most one of them may fall below the decision margin.
    compare_select(L, gpu, ref, label=label, dense_special_queries=c["dense_special"], criterion=c["criterion"],
                   capped=c["tau"] > 0, max_excluded=max(0.01, 1.0 / rows))
    q, k, v, _ = inputs
    o = ress.ress_sparse_attn(q, k, v, dev["kept_count"], dev["kept_idx"], bq=L.bq, bk=L.bk,
                              n_special_tail=L.n_special_tail)
    od = ress.ress_dense_attn(q, k, v, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail)
    torch.cuda.synchronize()
    hs, ts = np.meshgrid(np.arange(L.H), np.arange(L.N), indexing="ij")
    hs, ts = hs.ravel().astype(np.int32), ts.ravel().astype(np.int32)
    compare_attn(L, o, hs, ts, kept_count=gpu["kept_count"], kept_idx=gpu["kept_idx"], label=label + " sparse")
    compare_attn(L, od, hs, ts, label=label + " dense")


# Medium layers (4-12 views of 500-1400 patch tokens): larger budgets, so the
# restoration rounds swap many blocks at once; every selection row, attention on a
# stratified sample of tokens.
N_MEDIUM = 12


def draw_medium(n=N_MEDIUM, seed=35593):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        H = int(rng.integers(2, 5))
        cases.append(dict(views=int(rng.integers(4, 13)), patch=int(rng.integers(500, 1401)),
                          special=int(rng.choice([0, 1, 5])), H=H,
                          bq=int(rng.choice([64, 128])), bk=int(rng.choice([64, 128])),
                          sparsity=[round(float(x), 3) for x in rng.uniform(0.5, 0.95, size=H)],
                          rounds=int(rng.choice([1, 3, 5, 8])), criterion=int(rng.choice([0, 0, 1, 2])),
                          seed=int(rng.integers(0, 1 << 30))))
    return cases


MEDIUM = draw_medium()


@pytest.mark.parametrize("idx", range(N_MEDIUM))
def test_random_medium_layer(ress, idx):
    import torch

    from gpu_helpers import sample_tokens

    c = MEDIUM[idx]
    L = synth.make_layer(c["views"], c["patch"], c["special"], H=c["H"], bq=c["bq"], bk=c["bk"],
                         sparsity=np.asarray(c["sparsity"]), seed=c["seed"], name=f"medium{idx}")
    label = (f"medium {idx}: N={L.N} H={L.H} {L.bq}/{L.bk} special={L.n_special_tail} "
             f"budgets={L.budgets.tolist()} R={c['rounds']} criterion={c['criterion']}")
    say(f"[random layer] {label}")
    inputs = device_inputs(L)
    gpu, dev = gpu_select(L, inputs, rounds=c["rounds"], criterion=c["criterion"])
    ref = oracle_select(L, rounds=c["rounds"], criterion=c["criterion"])
    compare_select(L, gpu, ref, label=label, criterion=c["criterion"])
    q, k, v, _ = inputs
    o = ress.ress_sparse_attn(q, k, v, dev["kept_count"], dev["kept_idx"], bq=L.bq, bk=L.bk,
                              n_special_tail=L.n_special_tail)
    torch.cuda.synchronize()
    hs, ts = sample_tokens(L, 512, seed=idx)
    compare_attn(L, o, hs, ts, kept_count=gpu["kept_count"], kept_idx=gpu["kept_idx"], label=label + " sparse")

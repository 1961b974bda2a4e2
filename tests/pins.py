"""Pins of the CPU oracle: each check compares an oracle result with something
other than the oracle itself (a definition computed directly, a closed form, an
invariant, a library routine, or brute force). Every check raises AssertionError
on failure; test_oracle_pins.py runs them against the oracle and
test_oracle_mutations.py runs them against deliberately broken builds of it.
"""
from __future__ import annotations

import functools
import math

import numpy as np
from scipy.special import softmax

import direct
import oracle
import synth

EPS = 1e-4


@functools.lru_cache(maxsize=None)
def layer(name: str):
    if name == "forced":  # 20 key blocks of 64, the last two hold special tokens
        return synth.make_layer(6, 200, 5, H=2, block=64, sparsity=0.6, seed=7, name=name)
    if name == "plain":  # no special tokens, 12 key blocks of 32
        return synth.make_layer(4, 96, 0, H=2, block=32, sparsity=0.5, seed=8, name=name)
    if name == "brute":  # 13 key blocks, one forced: 12 candidates
        return synth.make_layer(2, 400, 8, H=2, block=64, sparsity=0.5, seed=9, name=name)
    if name == "ragged":  # partial last block, separate q / k block sizes
        return synth.make_layer(3, 150, 5, H=2, bq=64, bk=32, sparsity=0.7, seed=10, name=name)
    if name == "two":  # exactly two key blocks
        return synth.make_layer(1, 128, 0, H=2, block=64, sparsity=0.5, seed=11, name=name)
    raise KeyError(name)


@functools.lru_cache(maxsize=None)
def pooled(name: str):
    L = layer(name)
    return (direct.pool_numpy(L.q, L.bq), direct.pool_numpy(L.k, L.bk), direct.pool_numpy(L.v, L.bk))


def rows_of(name: str, step: int = 3):
    L = layer(name)
    return [(h, i) for h in range(L.H) for i in range(0, L.n_qb, step)]


def _row(name, h, i):
    L = layer(name)
    r = direct.row_inputs(L, h, i, pooled(name))
    r["W"] = L.w_o()[h]
    r["logits"] = direct.pooled_logits(r["qbar_i"], r["kbar"])
    return r


# --------------------------------------------------------------------------- pooling


def check_pool():
    for name in ("forced", "plain", "ragged"):
        L = layer(name)
        for x, b in ((L.q, L.bq), (L.k, L.bk), (L.v, L.bk)):
            np.testing.assert_allclose(oracle.pool(x, b), direct.pool_numpy(x, b), rtol=1e-14, atol=1e-15)


def check_forced():
    cases = [(43968, 128, 160, {342, 343}), (10992, 128, 40, {85}), (21984, 128, 80, {171}),
             (137400, 128, 500, set(range(1069, 1074))), (1024, 64, 0, set())]
    for N, bk, ns, expect in cases:
        got = set(np.flatnonzero(oracle.forced_blocks(N, bk, ns)).tolist())
        assert got == expect, (N, got, expect)
    for N, bk, ns in ((1230, 64, 30), (500, 32, 5), (128, 64, 128)):
        f = oracle.forced_blocks(N, bk, ns)
        for j in range(len(f)):
            toks = np.arange(j * bk, min((j + 1) * bk, N))
            assert f[j] == bool(np.any(toks >= N - ns)), (N, j)


# --------------------------------------------------------------------------- pooled map


def check_pooled_map():
    for name in ("forced", "plain", "ragged"):
        for h, i in rows_of(name):
            r = _row(name, h, i)
            P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
            ref = softmax(r["logits"])
            np.testing.assert_allclose(P, ref, rtol=1e-12, atol=1e-300)
            np.testing.assert_allclose(vb, ref @ r["vbar"], rtol=1e-11, atol=1e-14)


def check_single_mask():
    """Eqs. 3-4: masking one block changes the pooled output by P/(1-P) (vbar - V_j)."""
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 5):
            r = _row(name, h, i)
            P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
            for j in range(len(P)):
                drop = np.zeros(len(P), bool)
                drop[j] = True
                lhs = direct.drift_vec(r["logits"], r["vbar"], drop)
                rhs = P[j] / (1.0 - P[j]) * (vb - r["vbar"][j])
                np.testing.assert_allclose(lhs, rhs, rtol=1e-9, atol=1e-13)


# --------------------------------------------------------------------------- scores


def check_scores():
    """Eqs. 6 and 9: s_j = P_j ||W_O (vbar - V_j)|| with the materialised W_O."""
    for name in ("forced", "plain", "ragged"):
        for h, i in rows_of(name):
            r = _row(name, h, i)
            P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
            s, _ = oracle.scores_row(P, vb, r["vbar"], r["M"], EPS)
            ref = P * np.linalg.norm((vb[None, :] - r["vbar"]) @ r["W"].T, axis=1)
            np.testing.assert_allclose(s, ref, rtol=2e-6, atol=1e-300)


def check_key_singleton():
    """Eq. 7 and the reduction of Eq. 12 for a single dropped block: key_j^2 equals
    the squared projected change of the pooled output when only block j is masked."""
    for name in ("forced", "plain"):
        for h, i in rows_of(name):
            r = _row(name, h, i)
            P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
            _, key = oracle.scores_row(P, vb, r["vbar"], r["M"], EPS)
            for j in range(len(P)):
                if 1.0 - P[j] <= EPS:
                    continue
                drop = np.zeros(len(P), bool)
                drop[j] = True
                ref = direct.drift_sq_w(r["logits"], r["vbar"], r["W"], drop)
                np.testing.assert_allclose(key[j] ** 2, ref, rtol=4e-6, atol=1e-300)


def check_two_block():
    """Closed form with two key blocks: e_0 = P_1 (V_1 - V_0), so key_0 = P_0 ||W_O (V_1 - V_0)||
    and key_1 = P_1 ||W_O (V_1 - V_0)||: ReSS keeps the more probable block."""
    for h, i in rows_of("two", 1):
        r = _row("two", h, i)
        P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
        _, key = oracle.scores_row(P, vb, r["vbar"], r["M"], EPS)
        nrm = np.linalg.norm(r["W"] @ (r["vbar"][1] - r["vbar"][0]))
        np.testing.assert_allclose(key, P * nrm, rtol=2e-6)
        res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], np.zeros(2, np.uint8), 1,
                                rounds=3)
        assert res["kept"][int(np.argmax(P))] and res["kept"].sum() == 1


# --------------------------------------------------------------------------- objective


def _random_drops(cand, rng, n):
    idx = np.flatnonzero(cand)
    for _ in range(n):
        k = rng.integers(1, len(idx))
        drop = np.zeros(len(cand), bool)
        drop[rng.choice(idx, size=k, replace=False)] = True
        yield drop


def check_objective():
    """Eqs. 10-12: g/K is the change of the pooled output and J its squared
    projected norm, for arbitrary drop sets."""
    rng = np.random.default_rng(0)
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 4):
            r = _row(name, h, i)
            P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
            for drop in _random_drops(~r["forced"], rng, 12):
                J, g, K, G = oracle.objective(P, vb, r["vbar"], r["M"], drop, EPS)
                if K <= EPS:
                    continue
                np.testing.assert_allclose(g / K, direct.drift_vec(r["logits"], r["vbar"], drop),
                                           rtol=1e-9, atol=1e-13)
                np.testing.assert_allclose(J, direct.drift_sq_w(r["logits"], r["vbar"], r["W"], drop),
                                           rtol=4e-6)
                np.testing.assert_allclose(G, J * K * K, rtol=1e-12)


def check_deltas():
    """Eqs. 13-16: dJ_k is exactly J(D) - J(D with k restored or dropped)."""
    rng = np.random.default_rng(1)
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 5):
            r = _row(name, h, i)
            P, vb = oracle.pooled_row(r["qbar_i"], r["kbar"], r["vbar"])
            s, _ = oracle.scores_row(P, vb, r["vbar"], r["M"], EPS)
            cand = ~r["forced"]
            for drop in _random_drops(cand, rng, 4):
                J0 = direct.drift_sq_m(r["logits"], r["vbar"], r["M"], drop)
                dJ = oracle.deltas(P, s, vb, r["vbar"], r["M"], drop, cand, EPS)
                for k in np.flatnonzero(cand):
                    nd = drop.copy()
                    nd[k] = not nd[k]
                    if 1.0 - P[nd].sum() <= EPS:
                        continue
                    ref = J0 - direct.drift_sq_m(r["logits"], r["vbar"], r["M"], nd)
                    assert abs(dJ[k] - ref) <= 1e-9 * max(J0, 1e-300) + 1e-300, (name, h, i, k, dJ[k], ref)


# --------------------------------------------------------------------------- rounds


def _schedule(c, r):
    return max(1, math.floor(0.5 * c * 2.0 ** (-(r + 1))))


def check_schedule():
    """Eq. 17 with rho = 0.5, R = 5: about 0.484 c swaps in total, halving per round."""
    for c in (4, 8, 21, 42, 84, 172, 215):
        m = [oracle.swaps(c, 0.5, r, 1) for r in range(5)]
        assert m[0] == max(1, c // 4), (c, m)
        assert all(m[r + 1] <= m[r] for r in range(4)), (c, m)
        assert abs(sum(m) - 0.484375 * c) <= 5, (c, m)


def check_trajectory():
    """Every round restores the m blocks of D and drops the m blocks of S with the
    largest exact objective decrease at the round-start set (ties: lower index), and
    the recorded J of each stage is the drift of that stage's drop set."""
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 2):
            r = _row(name, h, i)
            cand = ~r["forced"]
            c = r["c"]
            res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=5)
            tD, tJ = res["trace_D"], res["trace_J"]
            Jm = lambda d: direct.drift_sq_m(r["logits"], r["vbar"], r["M"], d)
            single = np.array([Jm(np.eye(len(cand), dtype=bool)[j]) if cand[j] else -1.0
                               for j in range(len(cand))])
            kept0, gap0 = direct.top_by(single, cand, c)
            if gap0 > 1e-9 * single.max():
                assert np.array_equal(tD[0], cand & ~kept0), (name, h, i)
            n_p = cand.sum()
            for st in range(len(tD)):
                assert tD[st].sum() == n_p - c and not np.any(tD[st] & r["forced"])
                np.testing.assert_allclose(tJ[st], Jm(tD[st]), rtol=1e-9, atol=1e-300)
            for st in range(len(tD) - 1):
                Ds, Dn = tD[st], tD[st + 1]
                A, B = Ds & ~Dn, Dn & ~Ds
                m = min(_schedule(c, st), n_p - c, c)
                assert A.sum() == m and B.sum() == m, (name, h, i, st, A.sum(), m)
                Js = Jm(Ds)
                gain = np.full(len(cand), -np.inf)
                for k in np.flatnonzero(cand):
                    nd = Ds.copy()
                    nd[k] = not nd[k]
                    gain[k] = Js - Jm(nd)
                for chosen, member in ((A, Ds), (B, cand & ~Ds)):
                    ref, gap = direct.top_by(gain, member, m)
                    if gap > 1e-9 * Js:
                        assert np.array_equal(chosen, ref), (name, h, i, st)


def check_track_best():
    for name in ("forced", "plain", "ragged"):
        for h, i in rows_of(name, 2):
            r = _row(name, h, i)
            res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], r["c"], rounds=5)
            tJ, tD = res["trace_J"], res["trace_D"]
            best = int(np.argmin(tJ))  # first minimum
            assert res["J_best"] == tJ[best] and res["J_init"] == tJ[0]
            assert res["J_best"] <= res["J_init"]
            assert np.array_equal(res["kept"], r["forced"] | (~r["forced"] & ~tD[best]))


def check_ties():
    """Identical key/value blocks give equal probabilities and zero drift everywhere:
    every top-k falls back to the lower index, so the first c candidates are kept."""
    L = layer("forced")
    kb = np.repeat(pooled("forced")[1][0, :1], L.n_kb, axis=0)
    vb = np.repeat(pooled("forced")[2][0, :1], L.n_kb, axis=0)
    forced = np.zeros(L.n_kb, bool)
    forced[-2:] = True
    for c in (1, 4, 9):
        res = oracle.select_row(pooled("forced")[0][0, 3], kb, vb, L.gram[0].astype(np.float64),
                                forced, c, rounds=5)
        expect = forced.copy()
        expect[:c] = True
        assert np.array_equal(res["kept"], expect), (c, np.flatnonzero(res["kept"]))


def check_brute_force(report=None):
    """Eq. 2: the returned drop set is never better than the exact optimum and never
    worse than the initial selection."""
    L = layer("brute")
    for h in range(L.H):
        for i in range(0, L.n_qb, 2):
            r = _row("brute", h, i)
            cand = ~r["forced"]
            for c in (3, 6, 9):
                res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=5)
                jstar, _ = direct.brute_force_min(r["logits"], r["vbar"], r["M"], cand, c)
                jb = direct.drift_sq_m(r["logits"], r["vbar"], r["M"], cand & ~res["kept"])
                np.testing.assert_allclose(jb, res["J_best"], rtol=1e-9)
                assert jstar <= res["J_best"] * (1 + 1e-9)
                assert res["J_best"] <= res["J_init"]
                if report is not None:
                    report.append(res["J_best"] / jstar if jstar > 0 else 1.0)


def _direct_margin(r, c, criterion=0, cdf_tau=0.0, trace_D=None):
    """The decision margin of a row, from the definitions: the smallest relative
    gap of every cut the selection makes along its trajectory trace_D (the
    oracle's stages; each one is pinned separately by check_trajectory),
    computed from exact masked-softmax drifts rather than the closed forms:
      initial cut    gap between the c-th and (c+1)-th ranking value (key, P or
                     -key by criterion) over the largest |value|; with a CDF cap
                     also the distance of tau to the two partial masses around the
                     cut, over tau;
      each round     gap between the m-th and (m+1)-th exact single-swap gain
                     J(D) - J(D with k toggled) (negated when maximising), among
                     restores and among drops, over J(D);
      track-best     |J_new - J_best| / J_best whenever the new set differs from
                     the best one so far.
    Returns (margin, which) with which the kind of cut that attains it."""
    cand = ~r["forced"]
    n = len(cand)
    n_p = int(cand.sum())
    Jm = lambda d: direct.drift_sq_m(r["logits"], r["vbar"], r["M"], d)
    P = softmax(r["logits"])
    out = [(math.inf, "none")]
    if c >= n_p:
        return out[0]
    single = np.array([Jm(np.eye(n, dtype=bool)[j]) if cand[j] else 0.0 for j in range(n)])
    key = np.sqrt(single)  # Eq. 12 for a single dropped block: J({j}) = key_j^2
    rank = P if criterion == 1 else -key if criterion == 3 else key
    if criterion == 1 and cdf_tau > 0.0:
        mass = P[r["forced"]].sum()
        order = sorted(np.flatnonzero(cand).tolist(), key=lambda j: (-P[j], j))
        cnt = 0
        while cnt < len(order) and mass < cdf_tau:
            mass += P[order[cnt]]
            cnt += 1
        if 0 < cnt < c:
            out.append((min(mass - cdf_tau, cdf_tau - (mass - P[order[cnt - 1]])) / cdf_tau, "cdf"))
        lo = min(max(0, 2 - int(r["forced"].sum())), n_p)
        c = min(c, max(cnt, lo))
    if c > 0:
        _, gap = direct.top_by(rank, cand, c)
        vmax = np.abs(rank[cand]).max()
        out.append((gap / (vmax if vmax > 0 else 1e-300), "initial"))
    maximise = criterion in (2, 3)
    best_D = trace_D[0]
    best_J = Jm(best_D)
    for st in range(len(trace_D) - 1):
        Ds = trace_D[st]
        Js = Jm(Ds)
        m = min(_schedule(c, st), n_p - c, c)
        gain = np.full(n, -np.inf)
        for k in np.flatnonzero(cand):
            nd = Ds.copy()
            nd[k] = not nd[k]
            gain[k] = (Jm(nd) - Js) if maximise else (Js - Jm(nd))
        for member in (Ds, cand & ~Ds):
            _, gap = direct.top_by(gain, member, m)
            out.append((gap / (Js if Js > 0 else 1e-300), "round"))
        Dn = trace_D[st + 1]
        Jn = Jm(Dn)
        if not np.array_equal(Dn, best_D):
            out.append((abs(Jn - best_J) / (best_J if best_J > 0 else 1e-300), "track-best"))
        if (Jn > best_J) if maximise else (Jn < best_J):
            best_D, best_J = Dn, Jn
    return min(out, key=lambda t: t[0])


MARGIN_CASES = [(0, 0.0), (1, 0.0), (1, 0.5), (2, 0.0), (3, 0.0)]


def check_margin(report=None):
    """The oracle's decision margin (the gate of the bit-exact kept-list comparison
    against the GPU path) equals the margin recomputed from the definitions, for
    every criterion; exact ties give margin 0 and rows with nothing to decide
    give +inf."""
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 2):
            r = _row(name, h, i)
            P = softmax(r["logits"])
            if np.any(1.0 - P[~r["forced"]] <= EPS):
                continue  # the eps guard of Eq. 7 makes key^2 differ from the masked drift
            for crit, tau in MARGIN_CASES:
                res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], r["c"], rounds=5,
                                        criterion=crit, cdf_tau=tau)
                want, which = _direct_margin(r, r["c"], crit, tau, res["trace_D"])
                got = res["margin"]
                assert abs(got - want) <= 1e-7 * want + 1e-10, (name, h, i, crit, tau, got, want, which)
                if report is not None:
                    report.append((which, want))
    # Exact ties: identical blocks, every key and gain equal.
    L = layer("forced")
    kb = np.repeat(pooled("forced")[1][0, :1], L.n_kb, axis=0)
    vb = np.repeat(pooled("forced")[2][0, :1], L.n_kb, axis=0)
    forced = np.zeros(L.n_kb, bool)
    forced[-2:] = True
    for c in (1, 4, 9):
        res = oracle.select_row(pooled("forced")[0][0, 3], kb, vb, L.gram[0].astype(np.float64), forced, c, rounds=5)
        assert res["margin"] == 0.0, (c, res["margin"])
    # Nothing to decide: dense rows and full budgets.
    r = _row("forced", 0, 2)
    n_p = int((~r["forced"]).sum())
    for kw in (dict(c=n_p), dict(c=3, dense_row=True)):
        c = kw.pop("c")
        res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=5, **kw)
        assert res["margin"] == math.inf, (c, kw, res["margin"])


# --------------------------------------------------------------------------- other criteria
# (the paper's comparisons: probability selection and its CDF threshold, Table 2;
# drift maximisation, Fig. 8 / Sec. 6.1)


def check_probability_criterion():
    """Probability criterion: the kept candidates are the c largest pooled
    probabilities (softmax of the pooled logits, computed here), ties to the lower
    index; with rounds the stages still have exact drifts and track-best minimises."""
    for name in ("forced", "plain", "ragged"):
        for h, i in rows_of(name, 2):
            r = _row(name, h, i)
            cand, c = ~r["forced"], r["c"]
            P = softmax(r["logits"])
            res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=0,
                                    criterion=oracle.PROBABILITY)
            ref, gap = direct.top_by(P, cand, c)
            if gap > 1e-12:
                assert np.array_equal(res["kept"], r["forced"] | ref), (name, h, i)
            res5 = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=5,
                                     criterion=oracle.PROBABILITY)
            for st in range(len(res5["trace_D"])):
                np.testing.assert_allclose(res5["trace_J"][st],
                                           direct.drift_sq_m(r["logits"], r["vbar"], r["M"], res5["trace_D"][st]),
                                           rtol=1e-9, atol=1e-300)
            assert res5["J_best"] == res5["trace_J"].min() and res5["J_best"] <= res5["J_init"]
            assert res5["kept"].sum() == c + r["forced"].sum()


def check_cdf_threshold():
    """CDF cap on the probability criterion: the kept candidates are a prefix of the
    candidates in descending probability; unless the budget or the two-block floor
    binds, the kept mass (forced blocks included) reaches tau and dropping the last
    kept candidate would fall below it."""
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 2):
            r = _row(name, h, i)
            cand, c = ~r["forced"], r["c"]
            P = softmax(r["logits"])
            floor = max(0, 2 - int(r["forced"].sum()))
            for tau in (0.2, 0.5, 0.8, 0.95):
                res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=0,
                                        criterion=oracle.PROBABILITY, cdf_tau=tau)
                kept_c = res["kept"] & cand
                n = int(kept_c.sum())
                assert floor <= n <= c, (name, h, i, tau, n)
                ref, gap = direct.top_by(P, cand, n)
                if gap > 1e-12:
                    assert np.array_equal(kept_c, ref), (name, h, i, tau)
                mass = P[r["forced"]].sum() + P[kept_c].sum()
                smallest = P[kept_c].min() if n else 0.0
                if abs(mass - tau) > 1e-12 and abs(mass - smallest - tau) > 1e-12:
                    if floor < n < c:
                        assert mass >= tau and mass - smallest < tau, (name, h, i, tau, n, mass)
                    elif n == c:  # the budget binds: the prefix one shorter never reached tau
                        assert c == 0 or mass - smallest < tau, (name, h, i, tau, n, mass)


def check_drift_max():
    """Sign-flipped objective (Fig. 8, Sec. 6.1). Full flip with no rounds keeps the c
    smallest single-block drifts J({j}) = key_j^2; in the rounds every swap is the
    one that raises J most (at the round-start set), track-best keeps the largest J,
    and on small rows the result never exceeds the brute-force maximum."""
    for name in ("forced", "plain"):
        for h, i in rows_of(name, 2):
            r = _row(name, h, i)
            cand, c = ~r["forced"], r["c"]
            Jm = lambda d: direct.drift_sq_m(r["logits"], r["vbar"], r["M"], d)
            single = np.array([Jm(np.eye(len(cand), dtype=bool)[j]) if cand[j] else 0.0 for j in range(len(cand))])
            res0 = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=0,
                                     criterion=oracle.DRIFT_MAX_FULL)
            ref, gap = direct.top_by(-single, cand, c)
            if gap > 1e-9 * max(single.max(), 1e-300):
                assert np.array_equal(res0["kept"], r["forced"] | ref), (name, h, i)
            for crit in (oracle.DRIFT_MAX_SWAP, oracle.DRIFT_MAX_FULL):
                res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=5,
                                        criterion=crit)
                tD, tJ = res["trace_D"], res["trace_J"]
                best = int(np.argmax(tJ))  # first maximum
                assert res["J_best"] == tJ[best] and res["J_best"] >= res["J_init"]
                assert np.array_equal(res["kept"], r["forced"] | (cand & ~tD[best]))
                n_p = cand.sum()
                for st in range(len(tD) - 1):
                    Ds, Dn = tD[st], tD[st + 1]
                    A, B = Ds & ~Dn, Dn & ~Ds
                    m = min(_schedule(c, st), n_p - c, c)
                    assert A.sum() == m and B.sum() == m
                    Js = Jm(Ds)
                    rise = np.full(len(cand), -np.inf)
                    for k in np.flatnonzero(cand):
                        nd = Ds.copy()
                        nd[k] = not nd[k]
                        rise[k] = Jm(nd) - Js
                    for chosen, member in ((A, Ds), (B, cand & ~Ds)):
                        want, g2 = direct.top_by(rise, member, m)
                        if g2 > 1e-9 * Js:
                            assert np.array_equal(chosen, want), (name, h, i, st, crit)
    L = layer("brute")
    for h in range(L.H):
        for i in range(0, L.n_qb, 3):
            r = _row("brute", h, i)
            cand = ~r["forced"]
            for c in (3, 8):
                res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], c, rounds=5,
                                        criterion=oracle.DRIFT_MAX_FULL)
                jmax = direct.brute_force_max(r["logits"], r["vbar"], r["M"], cand, c)
                assert res["J_best"] <= jmax * (1 + 1e-9)


# --------------------------------------------------------------------------- driver


def _select_all(name, **kw):
    L = layer(name)
    return oracle.select(L.q, L.k, L.v, L.gram, L.budgets, N=L.N, bq=L.bq, bk=L.bk,
                         n_special=L.n_special_tail, **kw)


def check_select_driver():
    for name in ("forced", "plain", "ragged"):
        L = layer(name)
        out = _select_all(name, rounds=5)
        nf = synth.forced_block_count(L.N, L.bk, L.n_special_tail)
        for h in range(L.H):
            for i in range(L.n_qb):
                flat = h * L.n_qb + i
                r = _row(name, h, i)
                special = L.n_special_tail > 0 and min((i + 1) * L.bq, L.N) > L.N - L.n_special_tail
                res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], r["forced"], r["c"],
                                        rounds=5, dense_row=special)
                cnt = out["kept_count"][flat]
                lst = out["kept_idx"][flat]
                assert np.array_equal(lst[:cnt], np.flatnonzero(res["kept"]))
                assert np.all(lst[cnt:] == -1)
                assert cnt == (L.n_kb if special else int(L.budgets[h]) + nf)
                assert set(np.flatnonzero(r["forced"]).tolist()) <= set(lst[:cnt].tolist())
                assert out["drift"][flat, 1] == res["J_best"]


def check_edges():
    L = layer("forced")
    f = oracle.forced_blocks(L.N, L.bk, L.n_special_tail)
    r = _row("forced", 0, 2)
    res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], f, 0, rounds=5)
    assert np.array_equal(res["kept"], f) and res["J_best"] == res["J_init"]
    allf = np.ones(L.n_kb, bool)
    res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], allf, 0, rounds=5)
    assert res["kept"].all() and res["J_best"] == 0.0
    res = oracle.select_row(r["qbar_i"], r["kbar"][:1], r["vbar"][:1], r["M"], np.zeros(1, bool), 1)
    assert res["kept"].all()
    n_p = int((~f).sum())
    res = oracle.select_row(r["qbar_i"], r["kbar"], r["vbar"], r["M"], f, n_p, rounds=5)
    assert res["kept"].all() and res["J_best"] == 0.0


# --------------------------------------------------------------------------- attention


def _sdpa(L, kept_tok_mask=None):
    import torch

    q = torch.from_numpy(direct.decode(L.q))[None]
    k = torch.from_numpy(direct.decode(L.k))[None]
    v = torch.from_numpy(direct.decode(L.v))[None]
    m = None if kept_tok_mask is None else torch.from_numpy(kept_tok_mask)[None]
    return torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=m)[0].numpy()


def _token_mask(L, kept_count, kept_idx):
    H = L.H
    m = np.zeros((H, L.N, L.N), bool)
    kc = kept_count.reshape(H, L.n_qb)
    ki = kept_idx.reshape(H, L.n_qb, L.n_kb)
    for h in range(H):
        for i in range(L.n_qb):
            cols = np.zeros(L.N, bool)
            for j in ki[h, i, :kc[h, i]]:
                cols[j * L.bk:min((j + 1) * L.bk, L.N)] = True
            m[h, i * L.bq:min((i + 1) * L.bq, L.N)] = cols[None, :]
    return m


def check_attention():
    for name in ("plain", "ragged"):
        L = layer(name)
        hs, ts = np.meshgrid(np.arange(L.H), np.arange(L.N), indexing="ij")
        hs, ts = hs.ravel().astype(np.int32), ts.ravel().astype(np.int32)
        scale = 1.0 / math.sqrt(L.D)
        dense = oracle.attn_tokens(L.q, L.k, L.v, N=L.N, bq=L.bq, bk=L.bk, scale=scale, sel_h=hs, sel_t=ts)
        np.testing.assert_allclose(dense.reshape(L.H, L.N, L.D), _sdpa(L), rtol=1e-10, atol=1e-12)
        sel = _select_all(name, rounds=3)
        sp = oracle.attn_tokens(L.q, L.k, L.v, N=L.N, bq=L.bq, bk=L.bk, scale=scale, sel_h=hs, sel_t=ts,
                                kept_count=sel["kept_count"], kept_idx=sel["kept_idx"])
        mask = _token_mask(L, sel["kept_count"], sel["kept_idx"])
        np.testing.assert_allclose(sp.reshape(L.H, L.N, L.D), _sdpa(L, mask), rtol=1e-10, atol=1e-12)


def check_zero_sparsity():
    """With c_h = |P| nothing is dropped: the kept lists are every block and sparse
    attention equals dense attention exactly."""
    L = layer("forced")
    nf = synth.forced_block_count(L.N, L.bk, L.n_special_tail)
    full = np.full(L.H, L.n_kb - nf, np.int32)
    sel = oracle.select(L.q, L.k, L.v, L.gram, full, N=L.N, bq=L.bq, bk=L.bk, n_special=L.n_special_tail)
    assert np.all(sel["kept_count"] == L.n_kb) and np.all(sel["drift"] == 0.0)
    hs = np.repeat(np.arange(L.H), 64).astype(np.int32)
    ts = np.tile(np.linspace(0, L.N - 1, 64).astype(np.int32), L.H)
    scale = 1.0 / math.sqrt(L.D)
    dense = oracle.attn_tokens(L.q, L.k, L.v, N=L.N, bq=L.bq, bk=L.bk, scale=scale, sel_h=hs, sel_t=ts)
    sp = oracle.attn_tokens(L.q, L.k, L.v, N=L.N, bq=L.bq, bk=L.bk, scale=scale, sel_h=hs, sel_t=ts,
                            kept_count=sel["kept_count"], kept_idx=sel["kept_idx"])
    assert np.array_equal(dense, sp)


ALL = [check_pool, check_forced, check_pooled_map, check_single_mask, check_scores,
       check_key_singleton, check_two_block, check_objective, check_deltas, check_schedule,
       check_trajectory, check_track_best, check_ties, check_brute_force, check_select_driver,
       check_edges, check_attention, check_zero_sparsity, check_probability_criterion,
       check_cdf_threshold, check_drift_max, check_margin]

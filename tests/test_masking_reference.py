"""The oracle's single-block masking reference (Sec. 3, Fig. 2) and its rank
correlation, pinned to definitions computed independently here."""
import math

import numpy as np
import pytest
import scipy.stats

import oracle
import synth


def test_spearman_matches_scipy():
    rng = np.random.default_rng(5)
    for n in (2, 3, 17, 200):
        a = rng.normal(size=n)
        b = a + rng.normal(size=n)
        b[: n // 3] = np.round(b[: n // 3])  # ties
        a[1::4] = a[0]
        assert oracle.spearman(a, b) == pytest.approx(scipy.stats.spearmanr(a, b)[0], abs=1e-12, nan_ok=True)
    assert oracle.spearman([1, 2, 3, 4], [10, 20, 30, 40]) == pytest.approx(1.0)
    assert oracle.spearman([1, 2, 3, 4], [4, 3, 2, 1]) == pytest.approx(-1.0)
    assert math.isnan(oracle.spearman([1, 1, 1], [1, 2, 3]))


def _identity_change(L, h, i, j, scale):
    """Token-level form of Eqs. 3-4: removing block j from token t's softmax gives
    O_t(B minus j) - O_t(B) = pi/(1 - pi) (O_t - o_j), with pi the softmax mass of j
    and o_j the attention restricted to block j."""
    q = synth.bf16_bits_to_f32(L.q[h]).astype(np.float64)
    k = synth.bf16_bits_to_f32(L.k[h]).astype(np.float64)
    v = synth.bf16_bits_to_f32(L.v[h]).astype(np.float64)
    toks = np.arange(i * L.bq, min((i + 1) * L.bq, L.N))
    logits = scale * q[toks] @ k.T
    w = np.exp(logits - logits.max(1, keepdims=True))
    in_j = np.zeros(L.N, bool)
    in_j[j * L.bk:min((j + 1) * L.bk, L.N)] = True
    O = (w @ v) / w.sum(1, keepdims=True)
    pi = w[:, in_j].sum(1) / w.sum(1)
    o_j = (w[:, in_j] @ v[in_j]) / w[:, in_j].sum(1, keepdims=True)
    d = (pi / (1 - pi))[:, None] * (O - o_j)
    M = L.gram[h].astype(np.float64)
    return math.sqrt(np.einsum("td,de,te->", d, M, d))


def test_block_masking_change_matches_the_removal_identity():
    L = synth.make_layer(3, 100, 5, H=2, block=64, sparsity=0.5, seed=41, name="mask-ref")
    scale = 1 / math.sqrt(64)
    for h, i in ((0, 0), (1, 2), (1, L.n_qb - 1)):
        blocks = list(range(L.n_kb))
        got = oracle.block_masking_change(L.q, L.k, L.v, L.gram, N=L.N, bq=L.bq, bk=L.bk, scale=scale, h=h, i=i,
                                          blocks=blocks)
        ref = np.array([_identity_change(L, h, i, j, scale) for j in blocks])
        np.testing.assert_allclose(got, ref, rtol=1e-9, atol=1e-13)
        assert np.all(got > 0)


def test_product_rank_correlation_matches_the_oracle():
    """The package's row-wise Spearman (host code of the masking report) against
    the oracle's, including ties and a constant row."""
    from paper_2609_35593_amd import masking

    rng = np.random.default_rng(9)
    a = rng.normal(size=(4, 30))
    b = a + rng.normal(size=a.shape)
    b[:, :8] = np.round(b[:, :8])
    a[1, ::5] = a[1, 0]
    a[3] = 2.0
    got = masking.spearman_rows(a, b)
    for r in range(4):
        ref = oracle.spearman(a[r], b[r])
        assert (math.isnan(ref) and math.isnan(got[r])) or got[r] == pytest.approx(ref, abs=1e-12)


def test_block_drift_sq_is_the_projected_norm():
    """The per-block masking change: with M = I it is the plain squared norm, with
    the generator's M_h = W_O^h^T W_O^h it is ||W_O^h x||^2 with the materialised
    W_O^h (up to M_h's float32 rounding), summed over each block's tokens
    (partial last block included)."""
    rng = np.random.default_rng(3)
    H, N, bq = 2, 150, 64
    a = rng.standard_normal((H, N, 64)).astype(np.float32)
    b = rng.standard_normal((H, N, 64)).astype(np.float32)
    x = a.astype(np.float64) - b.astype(np.float64)
    eye = np.broadcast_to(np.eye(64, dtype=np.float32), (H, 64, 64))
    got = oracle.block_drift_sq(a, b, eye, bq=bq)
    want = np.array([[np.sum(x[h, i * bq:min((i + 1) * bq, N)] ** 2) for i in range(3)] for h in range(H)])
    np.testing.assert_allclose(got, want, rtol=1e-13)
    w, gram = synth.draw_w_o(H, 64, 11)
    got = oracle.block_drift_sq(a, b, gram, bq=bq)
    want = np.array([[np.sum((x[h, i * bq:min((i + 1) * bq, N)] @ w[h].T) ** 2) for i in range(3)] for h in range(H)])
    np.testing.assert_allclose(got, want, rtol=1e-6)


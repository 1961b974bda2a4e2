"""GPU parity of the fused projections on either side of the path, through the
C ABI, against the float64 oracle on the same seeded bf16 inputs.

Bar: |gpu - ref| <= ulp + K 2^-24 S for every output, where ref is the oracle's
once-rounded float64 result, ulp the bf16 spacing at max(|gpu|, |ref|), K the
reduction length and S = sum_k |a_k b_k| (the float32 accumulation error bound;
it only matters where the sum cancels to a small value), and at most 1% of
outputs differ at all (float32 sums round to the same bf16 value except next to
a rounding midpoint). The pooled state written by the QKV epilogue must give a
selection bit-identical to ress_select pooling the same Q, K, V itself.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ress():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_35593_amd as r

    return r


def _inputs(H, N, seed):
    rng = np.random.default_rng(seed)
    dm = 64 * H
    x = synth.f32_to_bf16_bits(rng.standard_normal((N, dm), dtype=np.float32))
    w_qkv = synth.f32_to_bf16_bits(rng.standard_normal((3 * dm, dm), dtype=np.float32) / np.float32(np.sqrt(dm)))
    w_o = synth.f32_to_bf16_bits(rng.standard_normal((dm, dm), dtype=np.float32) / np.float32(np.sqrt(dm)))
    resid = synth.f32_to_bf16_bits(rng.standard_normal((N, dm), dtype=np.float32))
    _, gram = synth.draw_w_o(H, 64, seed)
    return x, w_qkv, w_o, resid, gram


def _check(got_bits, ref_bits, acc_bound, label):
    g = synth.bf16_bits_to_f32(got_bits).astype(np.float64)
    r = synth.bf16_bits_to_f32(ref_bits).astype(np.float64)
    mag = np.maximum(np.maximum(np.abs(r), np.abs(g)), 2.0 ** -100)
    ulp = np.exp2(np.floor(np.log2(mag)) - 7)
    off = np.abs(g - r)
    frac = float(np.mean(off > 0))
    say(f"  {label}: {g.size} outputs, {frac:.3%} differ, max |d|/(ulp + bound) "
        f"{float((off / (ulp + acc_bound)).max()):.2f}")
    assert np.all(off <= (ulp + acc_bound) * (1 + 1e-12)), label
    assert frac <= 0.01, label


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def _qkv_bounds(x, w_qkv, H):
    """K 2^-24 sum_k |x_k w_k| for every output, in the head-major layout."""
    dm = 64 * H
    S = np.abs(_f64(x)) @ np.abs(_f64(w_qkv)).T * (dm * 2.0 ** -24)
    parts = S.reshape(len(x), 3, H, 64).transpose(1, 2, 0, 3)
    return parts[0], parts[1], parts[2]


CASES = [(4, 1000, 128, 128, 11), (4, 777, 64, 128, 12), (16, 2755, 128, 64, 13), (4, 1, 64, 64, 15),
         (8, 130, 128, 64, 16),
         # 768-wide model (3 output tiles per projection), token counts at and
         # around the 256-row tile edge
         (12, 255, 64, 64, 17), (12, 256, 128, 128, 18), (12, 257, 128, 64, 19), (8, 513, 64, 128, 20)]


@pytest.mark.parametrize("H,N,bq,bk,seed", CASES)
def test_qkv_projection_and_pooled_selection(ress, H, N, bq, bk, seed):
    import torch

    say(f"[qkv projection] H={H} N={N} bq={bq} bk={bk}")
    x, w_qkv, _, _, gram = _inputs(H, N, seed)
    dev = "cuda:0"
    gram_d = torch.from_numpy(gram).to(dev)
    out = ress.ress_qkv_proj_pool(ress.bf16_from_bits(x, dev), ress.bf16_from_bits(w_qkv, dev), gram_d, bq=bq, bk=bk)
    torch.cuda.synchronize()
    ref = oracle.qkv_projection(x, w_qkv, H)
    for name, r, bnd in zip("qkv", ref, _qkv_bounds(x, w_qkv, H)):
        got = out[name].view(torch.int16).cpu().numpy().view(np.uint16)
        _check(got, r, bnd, f"{name} H={H} N={N}")
    # The pooled state from the epilogue against ress_select pooling the same q, k, v.
    n_kb = (N + bk - 1) // bk
    budgets = np.full(H, min(n_kb, max(2, n_kb // 3)), np.int32)
    q, k, v = out["q"], out["k"], out["v"]
    fused = ress.ress_select(q, k, v, gram_d, budgets, bq=bq, bk=bk, want_debug=True, workspace=out["workspace"],
                             pooled_in_workspace=True)
    plain = ress.ress_select(q, k, v, gram_d, budgets, bq=bq, bk=bk, want_debug=True)
    torch.cuda.synchronize()
    for name in ("kept_count", "kept_idx", "drift", "key", "prob"):
        assert torch.equal(fused[name], plain[name]), name


def test_qkv_projection_32v_sampled(ress):
    """The full 32-view shape (43,968 tokens, model width 1024): sampled tokens of
    every head against the oracle, and the pooled selection against plain pooling."""
    import torch

    H, N = 16, 43968
    say(f"[qkv projection 32v] H={H} N={N}")
    x, w_qkv, _, _, gram = _inputs(H, N, 14)
    dev = "cuda:0"
    gram_d = torch.from_numpy(gram).to(dev)
    out = ress.ress_qkv_proj_pool(ress.bf16_from_bits(x, dev), ress.bf16_from_bits(w_qkv, dev), gram_d, bq=128,
                                  bk=128)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, 127, 128, N - 65, N - 64, N - 1],
                                     np.random.default_rng(5).integers(0, N, 57)]))
    ref = oracle.qkv_projection(x[rows], w_qkv, H)
    for name, r, bnd in zip("qkv", ref, _qkv_bounds(x[rows], w_qkv, H)):
        got = out[name][:, torch.from_numpy(rows)].view(torch.int16).cpu().numpy().view(np.uint16)
        _check(got, r, bnd, f"{name} 32v sampled")
    budgets = np.full(H, 84, np.int32)
    q, k, v = out["q"], out["k"], out["v"]
    fused = ress.ress_select(q, k, v, gram_d, budgets, bq=128, bk=128, workspace=out["workspace"],
                             pooled_in_workspace=True)
    plain = ress.ress_select(q, k, v, gram_d, budgets, bq=128, bk=128)
    torch.cuda.synchronize()
    for name in ("kept_count", "kept_idx", "drift"):
        assert torch.equal(fused[name], plain[name]), name


@pytest.mark.parametrize("H,N,seed", [(4, 1000, 21), (16, 2755, 22), (12, 257, 23), (8, 7, 24), (4, 256, 25)])
def test_out_projection_residual(ress, H, N, seed):
    import torch

    say(f"[out projection + residual] H={H} N={N}")
    _, _, w_o, resid, _ = _inputs(H, N, seed)
    o = synth.f32_to_bf16_bits(np.random.default_rng(seed + 100).standard_normal((H, N, 64), dtype=np.float32) * 0.3)
    dev = "cuda:0"
    o_d, w_d, r_d = (ress.bf16_from_bits(t, dev) for t in (o, w_o, resid))
    got = ress.ress_out_proj_residual(o_d, w_d, r_d)
    torch.cuda.synchronize()
    ref = oracle.out_projection_residual(o, w_o, resid)
    flat = np.abs(_f64(o)).transpose(1, 0, 2).reshape(N, 64 * H)
    bound = (flat @ np.abs(_f64(w_o)).T + np.abs(_f64(resid))) * ((64 * H + 1) * 2.0 ** -24)
    _check(got.view(torch.int16).cpu().numpy().view(np.uint16), ref, bound, f"residual H={H} N={N}")
    # in place: resid_out = resid_in
    ress.ress_out_proj_residual(o_d, w_d, r_d, resid_out=r_d)
    torch.cuda.synchronize()
    assert torch.equal(r_d, got)

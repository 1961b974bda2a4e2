"""The 24-layer stack (16 views, noise rising 0.3 -> 1.0 over the layers, 75%
sparsity) end to end on the device, with the change sparse attention makes to
what each layer adds to the residual stream accumulated in a float32 stream of
width 1024: r_L = sum_l W_O^l (O_sparse,l - O_dense,l) (Sec. 3, "The Right
Objective": the residual update x_{l+1} = x_l + f_l(x_l) carries the drift of
layer l into every later layer). Everything runs through the C ABI.

Bars:
  ress_out_proj_residual_f32  |gpu - ref| <= K 2^-24 S + 2^-23 |ref| per output
      against the float64 oracle (S = sum_k |a_k b_k| + |resid|, K = 1025).
  stream accumulation  on sampled tokens, r_L from the GPU equals the oracle's
      float64 sum over the layers of W_O^l applied to the GPU's own attention
      outputs, within the float32 accumulation bound summed over the 48 updates;
      those attention outputs (sparse and dense, every layer) are within the
      attention tolerance of the oracle's; the end-to-end difference of r_L to
      the stream built from the oracle's own attention is reported.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import ATTN_MAX, ATTN_MEAN, device_inputs, gpu_select, say, stack_layer, stack_w_o_bits

pytestmark = pytest.mark.gpu

K_BOUND = (1024 + 1) * 2.0 ** -24


@pytest.fixture(scope="module")
def ress():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_35593_amd as r

    return r


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


@pytest.mark.parametrize("H,N,seed", [(4, 1000, 41), (16, 2755, 42), (12, 257, 43), (8, 7, 44)])
def test_out_projection_residual_f32(ress, H, N, seed):
    import torch

    say(f"[out projection + float32 residual] H={H} N={N}")
    rng = np.random.default_rng(seed)
    dm = 64 * H
    o = synth.f32_to_bf16_bits(rng.standard_normal((H, N, 64), dtype=np.float32) * 0.3)
    w_o = synth.f32_to_bf16_bits(rng.standard_normal((dm, dm), dtype=np.float32) / np.float32(np.sqrt(dm)))
    resid = rng.standard_normal((N, dm), dtype=np.float32)
    dev = "cuda:0"
    o_d, w_d = ress.bf16_from_bits(o, dev), ress.bf16_from_bits(w_o, dev)
    r_d = torch.from_numpy(resid).to(dev)
    got = ress.ress_out_proj_residual_f32(o_d, w_d, r_d)
    torch.cuda.synchronize()
    rows = oracle.head_major_rows(o)
    ref = oracle.out_projection_f64(rows, w_o, resid)
    S = np.abs(rows) @ np.abs(_f64(w_o)).T + np.abs(resid)
    err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
    bound = K_BOUND * S + 2.0 ** -23 * np.abs(ref)
    say(f"  max |d|/bound {float((err / bound).max()):.3f}")
    assert np.all(err <= bound)
    ress.ress_out_proj_residual_f32(o_d, w_d, r_d, resid_out=r_d)  # in place
    torch.cuda.synchronize()
    assert torch.equal(r_d, got)


def test_residual_stream_16v_stack(ress):
    import torch

    dev = "cuda:0"
    L0 = stack_layer(0)
    H, N, dm = L0.H, L0.N, L0.H * L0.D
    # sampled tokens: first, last patch token, special tail, partial last block, uniform
    toks = np.unique(np.concatenate([[0, 1, 127, 128, N - L0.n_special_tail - 1, N - 1, N - 50],
                                     np.random.default_rng(7).integers(0, N, 33)])).astype(np.int64)
    r = torch.zeros((N, dm), dtype=torch.float32, device=dev)
    base = torch.zeros_like(r)
    ref_a = np.zeros((len(toks), dm))
    ref_b = np.zeros((len(toks), dm))
    bound = np.zeros((len(toks), dm))
    jmed = []
    tt = torch.from_numpy(toks)
    for layer in range(24):
        L = stack_layer(layer)
        w_bits = stack_w_o_bits(L)
        w = ress.bf16_from_bits(w_bits, dev)
        w_neg = ress.bf16_from_bits(w_bits ^ np.uint16(0x8000), dev)  # -W_O, exact
        inputs = device_inputs(L)
        q, k, v, _ = inputs
        sel, dsel = gpu_select(L, inputs, rounds=5, want_debug=False)
        o_s = ress.ress_sparse_attn(q, k, v, dsel["kept_count"], dsel["kept_idx"], bq=L.bq, bk=L.bk)
        o_d = ress.ress_dense_attn(q, k, v, bq=L.bq, bk=L.bk)
        ress.ress_out_proj_residual_f32(o_s, w, r, resid_out=r)
        ress.ress_out_proj_residual_f32(o_d, w_neg, r, resid_out=r)
        ress.ress_out_proj_residual_f32(o_d, w, base, resid_out=base)
        os_h = o_s[:, tt].float().cpu().numpy()
        od_h = o_d[:, tt].float().cpu().numpy()
        # (a) the stream from the GPU's own attention outputs, float64
        rs, rd = oracle.head_major_rows(os_h), oracle.head_major_rows(od_h)
        ref_a += oracle.out_projection_f64(rs, w_bits) - oracle.out_projection_f64(rd, w_bits)
        wa = np.abs(_f64(w_bits)).T
        bound += K_BOUND * (np.abs(rs) @ wa + np.abs(rd) @ wa)
        # (b) the oracle's own attention with the same kept lists
        hs = np.repeat(np.arange(H), len(toks)).astype(np.int32)
        ts = np.tile(toks, H).astype(np.int32)
        kc, ki = sel["kept_count"], sel["kept_idx"]
        a_s = oracle.attn_tokens(L.q, L.k, L.v, N=N, bq=L.bq, bk=L.bk, scale=0.125, sel_h=hs, sel_t=ts,
                                 kept_count=kc, kept_idx=ki).reshape(H, len(toks), 64)
        a_d = oracle.attn_tokens(L.q, L.k, L.v, N=N, bq=L.bq, bk=L.bk, scale=0.125, sel_h=hs,
                                 sel_t=ts).reshape(H, len(toks), 64)
        for got_o, ref_o, what in ((os_h, a_s, "sparse"), (od_h, a_d, "dense")):
            e = np.abs(got_o - ref_o)
            assert e.max() <= ATTN_MAX and e.mean() <= ATTN_MEAN, (layer, what, e.max(), e.mean())
        ref_b += oracle.out_projection_f64(oracle.head_major_rows(a_s) - oracle.head_major_rows(a_d), w_bits)
        dr = sel["drift"].reshape(-1, 2)
        live = dr[:, 0] > 0
        jmed.append(float(np.median(dr[live, 1])))
        del inputs, dsel, o_s, o_d
    torch.cuda.synchronize()
    got = r[tt].cpu().numpy().astype(np.float64)
    bound += 48 * 2.0 ** -24 * np.abs(ref_a) + 1e-30
    err_a = np.abs(got - ref_a)
    say(f"  stream vs float64 sum of the GPU's outputs: max |d|/bound {float((err_a / bound).max()):.3f}")
    assert np.all(err_a <= bound)
    rel_b = np.linalg.norm(got - ref_b) / np.linalg.norm(ref_b)
    drift = (torch.linalg.vector_norm(r) / torch.linalg.vector_norm(base)).item()
    say(f"  end to end vs the oracle's attention: relative norm error {rel_b:.3e}; "
        f"||r_L|| / ||sum_l W_O O_dense|| = {drift:.4f}; median J per layer {np.round(jmed, 5).tolist()}")
    assert np.all(np.isfinite(got)) and 0.0 < drift < 1.0


@pytest.mark.parametrize("H,N,bq", [(3, 1000, 128), (2, 150, 64), (16, 2755, 128)])
def test_block_drift_sq(ress, H, N, bq):
    """ress_block_drift_sq against the float64 oracle: the differences of float32
    values are exact in float64, so only the order of the float64 sums differs."""
    import torch

    say(f"[block drift sq] H={H} N={N} bq={bq}")
    rng = np.random.default_rng(H * 100 + bq)
    a = (rng.standard_normal((H, N, 64)) * 0.3).astype(np.float32)
    b = a + (rng.standard_normal((H, N, 64)) * 1e-3).astype(np.float32)
    _, gram = synth.draw_w_o(H, 64, 5)
    dev = "cuda:0"
    got = ress.ress_block_drift_sq(torch.from_numpy(a).to(dev), torch.from_numpy(b).to(dev),
                                   torch.from_numpy(gram).to(dev), bq=bq)
    torch.cuda.synchronize()
    ref = oracle.block_drift_sq(a, b, gram, bq=bq)
    np.testing.assert_allclose(got.cpu().numpy(), ref, rtol=1e-12, atol=0)


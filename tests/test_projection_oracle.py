"""The oracle's projections on either side of the path (QKV with its bf16
rounding, output projection + residual), pinned to cases with known answers."""
import numpy as np
import torch

import oracle
import synth


def test_bf16_rounding_is_nearest_even():
    # exactly representable values stay; halfway cases go to the even neighbour
    one = 1.0
    ulp = 2.0 ** -7  # bf16 spacing in [1, 2)
    vals = np.array([one, one + ulp, one + ulp / 2, one + 1.5 * ulp, -(one + ulp / 2), 3.0 * 2 ** -20,
                     one + ulp / 2 + 2 ** -30])
    got = synth.bf16_bits_to_f32(oracle.bf16_bits_nearest(vals)).astype(np.float64)
    np.testing.assert_array_equal(got, [one, one + ulp, one, one + 2 * ulp, -one, 3.0 * 2 ** -20, one + ulp])
    # agrees with torch's float32 -> bf16 rounding where float32 holds the value exactly
    x = np.random.default_rng(3).normal(size=4096).astype(np.float32)
    ref = torch.from_numpy(x).bfloat16().view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.bf16_bits_nearest(x.astype(np.float64)), ref)


def _bits(a):
    return synth.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def test_qkv_projection_identity_and_permutation():
    """With W_qkv = [I; 2I; P] (P a permutation), Q = x, K = 2x and V = x with
    its channels permuted, split into heads exactly."""
    H, N = 4, 37
    dm = 64 * H
    rng = np.random.default_rng(1)
    x = _bits(rng.normal(size=(N, dm)))
    perm = rng.permutation(dm)
    w = np.zeros((3 * dm, dm))
    w[:dm] = np.eye(dm)
    w[dm:2 * dm] = 2 * np.eye(dm)
    w[2 * dm + np.arange(dm), perm] = 1.0
    q, k, v = oracle.qkv_projection(x, _bits(w), H)
    xf = synth.bf16_bits_to_f32(x)
    for h in range(H):
        np.testing.assert_array_equal(synth.bf16_bits_to_f32(q[h]), xf[:, 64 * h:64 * h + 64])
        np.testing.assert_array_equal(synth.bf16_bits_to_f32(k[h]), 2 * xf[:, 64 * h:64 * h + 64])
        np.testing.assert_array_equal(synth.bf16_bits_to_f32(v[h]), xf[:, perm[64 * h:64 * h + 64]])


def test_qkv_projection_small_integers_are_exact():
    """Integer inputs and weights: every product and sum is exact, so the output is
    the integer matrix product (checked against an int64 product)."""
    H, N = 4, 20
    dm = 64 * H
    rng = np.random.default_rng(2)
    xi = rng.integers(-3, 4, size=(N, dm))
    wi = rng.integers(-2, 3, size=(3 * dm, dm))
    q, k, v = oracle.qkv_projection(_bits(xi), _bits(wi), H)
    y = xi @ wi.T  # |y| <= 3*2*256 = 1536 < 2^8 * 8: bf16 holds every value up to 256 exactly
    small = np.abs(y) <= 256
    got = np.concatenate([synth.bf16_bits_to_f32(t).transpose(1, 0, 2).reshape(N, dm) for t in (q, k, v)], 1)
    np.testing.assert_array_equal(got[small], y[small])
    assert small.mean() > 0.5


def test_out_projection_residual_cases():
    """W_O = I returns R + concat_h(O); W_O = 0 returns R; O from two heads of
    ones with W_O rows selecting one input channel give R + 1."""
    H, N = 4, 9
    dm = 64 * H
    rng = np.random.default_rng(4)
    o = _bits(rng.normal(size=(H, N, 64)))
    r = _bits(rng.normal(size=(N, dm)))
    flat = synth.bf16_bits_to_f32(o).astype(np.float64).transpose(1, 0, 2).reshape(N, dm)
    got = oracle.out_projection_residual(o, _bits(np.eye(dm)), r)
    np.testing.assert_array_equal(got, oracle.bf16_bits_nearest(synth.bf16_bits_to_f32(r).astype(np.float64) + flat))
    np.testing.assert_array_equal(oracle.out_projection_residual(o, _bits(np.zeros((dm, dm))), r), r)
    ones = _bits(np.ones((H, N, 64)))
    sel = np.zeros((dm, dm))
    sel[:, 70] = 1.0  # every output reads input channel 70 = head 1, channel 6
    zero_r = _bits(np.zeros((N, dm)))
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(oracle.out_projection_residual(ones, _bits(sel), zero_r)),
                                  np.ones((N, dm), np.float32))


def test_out_projection_f64_cases():
    """The float64 stream update: W_O = I returns R + concat_h(O) exactly; W_O = 0
    returns R; a permutation W_O permutes the channels; -W_O cancels W_O; small
    integers give the exact integer product; head_major_rows lays heads out as
    channel 64h + d."""
    H, N = 4, 11
    dm = 64 * H
    rng = np.random.default_rng(5)
    o = _bits(rng.normal(size=(H, N, 64)))
    r = rng.normal(size=(N, dm)).astype(np.float32)
    rows = oracle.head_major_rows(o)
    of = synth.bf16_bits_to_f32(o).astype(np.float64)
    for h in range(H):
        np.testing.assert_array_equal(rows[:, 64 * h:64 * h + 64], of[h])
    np.testing.assert_array_equal(oracle.head_major_rows(o, [3, 7]), rows[[3, 7]])
    np.testing.assert_array_equal(oracle.out_projection_f64(rows, _bits(np.eye(dm)), r), r.astype(np.float64) + rows)
    np.testing.assert_array_equal(oracle.out_projection_f64(rows, _bits(np.zeros((dm, dm))), r), r)
    perm = rng.permutation(dm)
    pm = np.zeros((dm, dm))
    pm[np.arange(dm), perm] = 1.0
    np.testing.assert_array_equal(oracle.out_projection_f64(rows, _bits(pm)), rows[:, perm])
    w = _bits(rng.normal(size=(dm, dm)) / 16)
    neg = w ^ np.uint16(0x8000)
    np.testing.assert_array_equal(oracle.out_projection_f64(rows, w) + oracle.out_projection_f64(rows, neg), 0.0)
    oi = rng.integers(-3, 4, size=(N, dm))
    wi = rng.integers(-2, 3, size=(dm, dm))
    np.testing.assert_array_equal(oracle.out_projection_f64(oi.astype(np.float64), _bits(wi)), oi @ wi.T)


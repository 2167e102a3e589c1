"""Pins of the oracle's INT4 round-to-nearest (group 64) AdaLN weight layer: hand-computed codes
and scales (including ties), the round-to-nearest error bound, exact reconstruction of weights
that lie on the grid, sign symmetry, zero groups, packing bytes, a closed-form layer output, and
the noise level of 4-bit RTN on Gaussian weights."""

import numpy as np

import oracle


def _row(vals, K=64):
    W = np.zeros((1, K))
    W[0, :len(vals)] = vals
    return W


def test_hand_computed_group():
    # absmax 3.5 -> scale 3.5 / 7 = 0.5 exactly; -1.75 / 0.5 = -3.5 and 0.25 / 0.5 = 0.5 are ties
    # that go to the even neighbour (-4 and 0); 1.25 / 0.5 = 2.5 -> 2; 0.75 / 0.5 = 1.5 -> 2
    q, s = oracle.rtn_int4_quantize(_row([3.5, -1.75, 0.25, 1.25, 0.75, -3.5, 0.0, 1.0]))
    assert s.tolist() == [[0.5]]
    assert q[0, :8].tolist() == [7, -4, 0, 2, 2, -7, 0, 2]
    assert not q[0, 8:].any()


def test_scale_is_fp16_of_the_fp32_quotient():
    # absmax 1.0: 1/7 in fp32 is 0.142857149..., whose fp16 rounding is 0.142822265625
    q, s = oracle.rtn_int4_quantize(_row([1.0, 0.5]))
    assert s[0, 0] == 0.142822265625
    assert q[0, 0] == 7 and q[0, 1] == 4          # 0.5 / 0.1428 = 3.5008... -> 4


def test_round_to_nearest_error_bound_and_symmetry():
    rng = np.random.default_rng(0)
    W = oracle.bf16_round(rng.standard_normal((40, 256)) * 0.02)
    q, s = oracle.rtn_int4_quantize(W)
    err = np.abs(W - oracle.rtn_int4_dequantize(q, s))
    assert np.all(err <= np.repeat(s, 64, axis=1) * (0.5 + 1e-6))
    assert q.min() >= -7 and q.max() <= 7
    q2, s2 = oracle.rtn_int4_quantize(-W)
    assert np.array_equal(s2, s) and np.array_equal(q2, -q)


def test_grid_weights_reconstruct_exactly():
    rng = np.random.default_rng(1)
    k = rng.integers(-7, 8, size=(8, 128))
    k[:, 0] = 7
    k[:, 64] = -7                                  # every group reaches its absmax
    W = k * 2.0 ** -6
    q, s = oracle.rtn_int4_quantize(W)
    assert np.all(s == 2.0 ** -6)
    assert np.array_equal(q, k) and np.array_equal(oracle.rtn_int4_dequantize(q, s), W)


def test_zero_group_has_zero_scale_and_codes():
    W = np.zeros((2, 128))
    W[1, 64:] = 0.01
    q, s = oracle.rtn_int4_quantize(W)
    assert s[0].tolist() == [0.0, 0.0] and s[1, 0] == 0.0 and s[1, 1] > 0
    assert not q[0].any() and not q[1, :64].any() and np.all(q[1, 64:] == 7)


def test_pack_bytes_and_roundtrip():
    q = np.array([[-8, 7, 0, -1]], dtype=np.int8)
    assert oracle.pack_rtn_int4(q).tolist() == [[0xF0, 0x78]]    # nibbles 0, 15 | 8, 7
    rng = np.random.default_rng(2)
    q = rng.integers(-8, 8, size=(5, 192)).astype(np.int8)
    assert np.array_equal(oracle.unpack_rtn_int4(oracle.pack_rtn_int4(q), 192), q)


def test_linear_closed_form():
    # every weight 3 * 2^-5 (scale 3 * 2^-5 / 7 rounds; code 7); X rows constant c_m -> Y = K c_m 7 s
    K = 192
    W = np.full((5, K), 3 * 2.0 ** -5)
    q, s = oracle.rtn_int4_quantize(W)
    X = np.array([[1.0] * K, [-2.0] * K])
    Y = oracle.rtn_int4_linear(X, q, s, bias=np.arange(5.0))
    want = np.outer([1.0, -2.0], np.full(5, K * 7 * s[0, 0])) + np.arange(5.0)
    assert np.allclose(Y, want, rtol=1e-15, atol=0)


def test_gaussian_weight_noise_level():
    # 4-bit symmetric RTN on N(0, 1) groups of 64: step = absmax / 7 (absmax ~ 2.4), uniform rounding
    # noise of rms step / sqrt(12) ~ 0.1 of the weights; a random-input layer inherits that ratio
    rng = np.random.default_rng(3)
    W = rng.standard_normal((512, 1024))
    X = rng.standard_normal((16, 1024))
    q, s = oracle.rtn_int4_quantize(W)
    rel_w = np.linalg.norm(W - oracle.rtn_int4_dequantize(q, s)) / np.linalg.norm(W)
    rel_y = np.linalg.norm(X @ W.T - oracle.rtn_int4_linear(X, q, s)) / np.linalg.norm(X @ W.T)
    assert 0.08 < rel_w < 0.12 and 0.08 < rel_y < 0.12

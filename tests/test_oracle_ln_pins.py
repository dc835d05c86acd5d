"""Pins for the oracle's LayerNorm-fused quantizer (ln_quantize_act and
layernorm_stats), none of which re-types the oracle's own formula:

* hand-worked rows whose mean and variance are known in closed form;
* numpy's float64 mean and population variance (an independent library
  routine) on random rows, incl. large and subnormal fp16 values;
* a hand-worked example through every per-element step (ties included);
* the textbook float64 LayerNorm followed by Eq. (g)'s quantization, which
  must give the same codes except within a hair of a rounding tie;
* invariants: scaling a row by a power of two (eps = 0) leaves every code
  unchanged; a constant row quantizes its shifted bias alone.

test_oracle_ln_mutations plants mistakes in the oracle and checks these fail.
"""
import numpy as np
import pytest

from oracle import ot_oracle as O


def test_stats_closed_form_rows():
    H = np.array([[1, 3, 1, 3], [0, 0, 0, 4], [5, 5, 5, 5], [-2, 2, -2, 2]], dtype=np.float16)
    mean, var = O.layernorm_stats(H)
    assert mean.tolist() == [2.0, 1.0, 5.0, 0.0]
    # population variance (divisor K): 1, 3, 0, 4
    assert var.tolist() == [1.0, 3.0, 0.0, 4.0]


@pytest.mark.parametrize("scale", [1e-6, 1.0, 300.0, 5e3])
def test_stats_match_numpy_float64(scale):
    r = np.random.default_rng(7)
    H = (r.standard_normal((6, 1040)) * scale + 0.3 * scale).astype(np.float16)
    mean, var = O.layernorm_stats(H)
    h = H.astype(np.float64)
    ref_m, ref_v = h.mean(axis=1), h.var(axis=1)
    assert np.all(np.abs(mean - ref_m) <= 1e-14 * np.abs(h).max(axis=1))
    assert np.all(np.abs(var - ref_v) <= 1e-12 * ref_v)


def _ones(K):
    return np.ones(K, dtype=np.float16)


def test_hand_worked_example_every_step():
    # row [-1, 1, -1, 1]: mean 0, variance 1; eps 0 gives rstd 1 exactly
    H = np.array([[-1, 1, -1, 1]], dtype=np.float16)
    gamma = np.array([1, 2, 1, 0.5], dtype=np.float16)
    beta = np.array([0, 0, 1, 0], dtype=np.float16)
    z = np.array([0, 0, 0.5, 0], dtype=np.float32)
    inv_s = np.full(4, 2.0, dtype=np.float32)
    # n = [-1, 1, -1, 1]; g = [-1, 2, -1, 0.5]; c = beta - z = [0, 0, 0.5, 0]
    # y = [-1, 2, -0.5, 0.5]; u = [-2, 4, -1, 1]
    q = O.ln_quantize_act(H, gamma, beta, 0.0, z, inv_s, 8)
    assert q.tolist() == [[-2, 4, -1, 1]]
    # ties: c = 0.25 gives y = -0.75, 1.25 -> u = -1.5, 2.5 -> -2, 2 (half to even)
    q = O.ln_quantize_act(H, _ones(4), np.full(4, 0.25, np.float16), 0.0,
                          np.zeros(4, np.float32), inv_s, 8)
    assert q.tolist() == [[-2, 2, -2, 2]]
    # clamp: u = +-100 with 6-bit codes -> +-31
    q = O.ln_quantize_act(H, _ones(4), np.zeros(4, np.float16), 0.0, np.zeros(4, np.float32),
                          np.full(4, 100.0, np.float32), 6)
    assert q.tolist() == [[-31, 31, -31, 31]]
    # eps: variance 1 and eps 3 give rstd 1/2 -> n = +-0.5 -> u = +-1
    q = O.ln_quantize_act(H, _ones(4), np.zeros(4, np.float16), 3.0, np.zeros(4, np.float32),
                          inv_s, 8)
    assert q.tolist() == [[-1, 1, -1, 1]]


def _textbook(H, gamma, beta, eps, z, s, a_bits):
    """fp64 LayerNorm (numpy mean/var), symmetrize, divide by s, unrounded."""
    h = H.astype(np.float64)
    y = (h - h.mean(1, keepdims=True)) / np.sqrt(h.var(1, keepdims=True) + float(np.float32(eps)))
    y = y * gamma.astype(np.float64) + beta.astype(np.float64)
    return (y - z.astype(np.float64)) / s.astype(np.float64)


@pytest.mark.parametrize("a_bits", [8, 6])
def test_codes_match_textbook_layernorm_then_quantize(a_bits):
    r = np.random.default_rng(11)
    M, K = 24, 768
    H = (r.standard_normal((M, K)) * 4 + r.uniform(-3, 3, K)).astype(np.float16)
    gamma = r.uniform(0.5, 2.0, K).astype(np.float16)
    beta = r.normal(0, 0.5, K).astype(np.float16)
    z = r.normal(0, 0.5, K).astype(np.float32)
    s = (r.uniform(0.05, 0.1, K) * (127 / O.qmax(a_bits))).astype(np.float32)
    inv_s = (1.0 / s.astype(np.float64)).astype(np.float32)
    q = O.ln_quantize_act(H, gamma, beta, 1e-5, z, inv_s, a_bits)
    u = _textbook(H, gamma, beta, 1e-5, z, s, a_bits)
    qa = O.qmax(a_bits)
    ref = np.clip(np.rint(u), -qa, qa)
    near_tie = np.abs(np.abs(u - np.trunc(u)) - 0.5) < 1e-4
    differ = q != ref
    assert np.all(np.abs(q.astype(int) - ref) <= 1)
    assert not np.any(differ & ~near_tie)
    assert (np.abs(u) < qa).mean() > 0.9  # most codes are unclipped


def test_power_of_two_scaling_leaves_codes_unchanged():
    r = np.random.default_rng(5)
    H = (r.standard_normal((8, 512)) * 3).astype(np.float16)
    gamma = r.uniform(0.5, 2, 512).astype(np.float16)
    beta = r.normal(0, 1, 512).astype(np.float16)
    z = r.normal(0, 1, 512).astype(np.float32)
    inv_s = r.uniform(5, 20, 512).astype(np.float32)
    q = O.ln_quantize_act(H, gamma, beta, 0.0, z, inv_s, 8)
    for k in (-3, 1, 4):
        Hk = (H.astype(np.float64) * 2.0 ** k).astype(np.float16)
        assert np.array_equal(Hk.astype(np.float64), H.astype(np.float64) * 2.0 ** k)
        assert np.array_equal(O.ln_quantize_act(Hk, gamma, beta, 0.0, z, inv_s, 8), q)


def test_constant_row_quantizes_the_shifted_bias():
    K = 64
    r = np.random.default_rng(9)
    beta = r.normal(0, 1, K).astype(np.float16)
    z = r.normal(0, 1, K).astype(np.float32)
    inv_s = r.uniform(5, 20, K).astype(np.float32)
    gamma = r.uniform(0.5, 2, K).astype(np.float16)
    want = np.clip(np.rint((beta.astype(np.float64) - z) * inv_s), -127, 127)
    for v in (0.0, 3.5, -1000.0):
        H = np.full((2, K), v, dtype=np.float16)
        q = O.ln_quantize_act(H, gamma, beta, 1e-5, z, inv_s, 8)
        u = (beta.astype(np.float64) - z) * inv_s
        ok = np.abs(np.abs(u - np.trunc(u)) - 0.5) > 1e-4
        assert np.array_equal(q[0][ok], want[ok]) and np.array_equal(q[0], q[1])

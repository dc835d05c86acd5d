"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

None of these re-types the oracle's formulas: each check is a hand-worked
example, an exact identity that holds only if every step is right, a
brute-force definition, an invariant, or a bound derived from Eq. (f)/(g).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import ot_oracle as O
from paper_2406_18832_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# Hand-worked example (tests/golden/hand_w3a3.json)
# --------------------------------------------------------------------------
def test_hand_worked_example_every_stage():
    g = _load("hand_w3a3.json")
    batches = [np.array(b, dtype=np.float16) for b in g["calib_batches"]]
    minmax, z, s, inv_s = O.calibrate(batches, g["a_bits"])
    np.testing.assert_array_equal(minmax, np.float32(g["minmax"]))
    np.testing.assert_array_equal(z, np.float32(g["z"]))
    np.testing.assert_array_equal(s, np.float32(g["s"]))
    np.testing.assert_array_equal(inv_s, np.float32(g["inv_s"]))

    W = np.array(g["W"], dtype=np.float16)
    b = np.array(g["b"], dtype=np.float16)
    Wq, sW, bprime = O.fold_weights(W, b, z, s, g["w_bits"])
    np.testing.assert_array_equal(Wq, np.int8(g["Wq"]))
    np.testing.assert_array_equal(sW, np.float32(g["sW"]))
    np.testing.assert_array_equal(bprime, np.float32(g["bprime"]))

    X = np.array(g["X"], dtype=np.float16)
    Xq = O.quantize_act(X, z, inv_s, g["a_bits"])
    np.testing.assert_array_equal(Xq, np.int8(g["Xq"]))
    acc = O.int_gemm(Xq, Wq)
    np.testing.assert_array_equal(acc, np.int32(g["acc"]))
    Y = O.epilogue(acc, sW, bprime)
    np.testing.assert_array_equal(Y, np.float16(g["Y"]))


# --------------------------------------------------------------------------
# Rounding disabled: the fold must reproduce X W^T + b exactly
# --------------------------------------------------------------------------
def _dyadic_problem(seed, M, K, N, a_bits, w_bits):
    """Inputs on which no step of the method rounds.

    Channel k is calibrated on [c_k - qa 2^e_k, c_k + qa 2^e_k], so s_k = 2^e_k
    and z_k = c_k exactly; activations are c_k + j 2^e_k with integer |j|<=qa,
    so their codes are j.  Weight row n is m_nk 2^f_n / s_k with integer
    |m_nk| <= qw (one entry of each row equal to qw), so the folded row is
    m_n 2^f_n, its scale is 2^f_n and its codes are m_n.  Then every float
    operation of the pipeline is exact, and the quantized linear must equal
    X W^T + b to the last bit.
    """
    r = np.random.default_rng(seed)
    qa, qw = O.qmax(a_bits), O.qmax(w_bits)
    e = r.integers(-3, 2, size=K)
    c = r.integers(-8, 9, size=K) * 0.25
    s = np.exp2(e.astype(np.float64))
    lo = c - qa * s
    hi = c + qa * s
    calib = [np.stack([lo, hi, c]).astype(np.float16)]
    j = r.integers(-qa, qa + 1, size=(M, K))
    X = (c[None, :] + j * s[None, :]).astype(np.float16)
    f = r.integers(-8, -4, size=N)
    m = r.integers(-qw, qw + 1, size=(N, K))
    m[np.arange(N), r.integers(0, K, size=N)] = qw
    W = (m * np.exp2(f.astype(np.float64))[:, None] / s[None, :]).astype(np.float16)
    b = (r.integers(-16, 17, size=N) * 0.125).astype(np.float16)
    # the construction itself must be exact in fp16
    assert np.all(X.astype(np.float64) == c[None, :] + j * s[None, :])
    assert np.all(W.astype(np.float64) * s[None, :] == m * np.exp2(f.astype(np.float64))[:, None])
    return calib, X, W, b, j, m


@pytest.mark.parametrize("a_bits,w_bits", [(8, 8), (6, 6), (8, 4)])
def test_rounding_free_fold_reproduces_linear_exactly(a_bits, w_bits):
    M, K, N = 7, 40, 9  # N != K so a transposed operand cannot pass
    calib, X, W, b, j, m = _dyadic_problem(11 + a_bits, M, K, N, a_bits, w_bits)
    minmax, z, s, inv_s = O.calibrate(calib, a_bits)
    Wq, sW, bprime = O.fold_weights(W, b, z, s, w_bits)
    Xq = O.quantize_act(X, z, inv_s, a_bits)
    np.testing.assert_array_equal(Xq, j)
    np.testing.assert_array_equal(Wq, m)
    acc = O.int_gemm(Xq, Wq)
    y = O.epilogue_fp32(acc, sW, bprime)
    exact = O.reference_fp64(X, W, b)
    np.testing.assert_array_equal(y.astype(np.float64), exact)


# --------------------------------------------------------------------------
# Integer GEMM: textbook triple loop on tiny shapes
# --------------------------------------------------------------------------
@pytest.mark.parametrize("M,K,N", [(1, 16, 1), (3, 32, 5), (5, 48, 2)])
def test_int_gemm_matches_triple_loop(M, K, N):
    r = np.random.default_rng(M * 100 + K + N)
    Xq = r.integers(-127, 128, size=(M, K)).astype(np.int8)
    Wq = r.integers(-127, 128, size=(N, K)).astype(np.int8)
    acc = O.int_gemm(Xq, Wq)
    for i in range(M):
        for n in range(N):
            ref = 0
            for k in range(K):
                ref += int(Xq[i, k]) * int(Wq[n, k])
            assert acc[i, n] == ref


def test_int_gemm_extreme_codes_stay_exact():
    # all-extreme codes: every partial sum is a multiple of 127^2, the largest
    # the method can produce at this K
    K = 4096
    Xq = np.full((2, K), 127, dtype=np.int8)
    Xq[1] = -127
    Wq = np.full((3, K), 127, dtype=np.int8)
    Wq[2, ::2] = -127
    acc = O.int_gemm(Xq, Wq)
    assert acc[0, 0] == K * 127 * 127 and acc[1, 0] == -K * 127 * 127
    assert acc[0, 2] == 0


def test_acc_range_guard():
    # 133144 * 127^2 = 2147479576 < 2^31 <= 133145 * 127^2
    O.check_acc_range(133144, 8, 8)
    with pytest.raises(OverflowError):
        O.check_acc_range(133145, 8, 8)
    # 2234634 * 31^2 = 2147483274 < 2^31 <= 2234635 * 31^2
    O.check_acc_range(2234634, 6, 6)
    with pytest.raises(OverflowError):
        O.check_acc_range(2234635, 6, 6)


# --------------------------------------------------------------------------
# Calibration (Sec. 3.2, App. A)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("a_bits", [8, 6])
def test_calibration_extremes_map_to_full_range(a_bits):
    wl = synth.WORKLOADS["opt125m_w8a8"]
    batches = list(synth.calibration_batches(wl, 0))
    minmax, z, s, inv_s = O.calibrate(batches, a_bits)
    qa = O.qmax(a_bits)
    allx = np.concatenate(batches)
    q = O.quantize_act(allx, z, inv_s, a_bits)
    assert q.min() >= -qa and q.max() <= qa
    # every non-constant channel reaches both ends of the code range
    nonconst = allx.max(axis=0) != allx.min(axis=0)
    assert nonconst.all()
    np.testing.assert_array_equal(q.max(axis=0), qa)
    np.testing.assert_array_equal(q.min(axis=0), -qa)
    # z is the midpoint of the range, s its half-width over qa (Sec. 3.2)
    lo = allx.min(axis=0).astype(np.float64)
    hi = allx.max(axis=0).astype(np.float64)
    np.testing.assert_allclose(hi - z, z - lo, rtol=0, atol=1e-5 * np.abs(hi - lo).max())
    np.testing.assert_allclose(s.astype(np.float64) * qa * 2, hi - lo, rtol=2 ** -23)
    np.testing.assert_array_equal(minmax, np.concatenate([lo, hi]).astype(np.float32))


def test_calibration_is_order_independent_and_streams():
    wl = synth.WORKLOADS["opt125m_w8a8"]
    batches = list(synth.calibration_batches(wl, 0))
    one = O.calibrate([np.concatenate(batches)], 8)
    rev = O.calibrate(batches[::-1], 8)
    for a, b in zip(one, rev):
        np.testing.assert_array_equal(a, b)


def test_constant_channel_gets_unit_scale_and_zero_codes():
    x = np.array([[3.0, 1.0], [3.0, -1.0]], dtype=np.float16)
    _, z, s, inv_s = O.calibrate([x], 8)
    assert s[0] == 1.0 and z[0] == 3.0 and inv_s[0] == 1.0
    q = O.quantize_act(np.array([[3.0, 0.0]], dtype=np.float16), z, inv_s, 8)
    assert q[0, 0] == 0


def test_negative_zero_is_plus_zero():
    x = np.array([[-0.0, 0.0], [-0.0, -0.0]], dtype=np.float16)
    minmax, z, s, _ = O.calibrate([x], 8)
    assert not np.any(np.signbit(minmax)) and not np.any(np.signbit(z))


@pytest.mark.parametrize("bad", [np.inf, -np.inf, np.nan])
def test_non_finite_calibration_rejected(bad):
    x = np.zeros((3, 4), dtype=np.float16)
    x[1, 2] = bad
    with pytest.raises(O.NonFinite):
        O.calibrate([x], 8)


# --------------------------------------------------------------------------
# Weight fold (Eq. (e), (f), (g))
# --------------------------------------------------------------------------
@pytest.mark.parametrize("w_bits", [8, 6])
def test_fold_invariants(w_bits):
    wl = synth.WORKLOADS["opt125m_w8a8"]
    _, z, s, _ = O.calibrate(list(synth.calibration_batches(wl, 0)), 8)
    W = synth.weight(wl, 0)
    b = synth.bias(wl, 0)
    Wq, sW, bprime = O.fold_weights(W, b, z, s, w_bits)
    qw = O.qmax(w_bits)
    Ws = W.astype(np.float64) * s.astype(np.float64)[None, :]
    # the fold is exact: dividing the folded weight by s gives W back (Eq. (e))
    np.testing.assert_array_equal(Ws / s.astype(np.float64)[None, :], W.astype(np.float64))
    # each row's largest folded weight lands on +-qw, everything within range
    am = np.abs(Ws).argmax(axis=1)
    np.testing.assert_array_equal(np.abs(Wq[np.arange(W.shape[0]), am]), qw)
    assert np.abs(Wq.astype(np.int32)).max() <= qw
    # round-to-nearest: |Wq sW - Ws| <= sW / 2 (up to the fp32 scale rounding)
    err = np.abs(Wq * sW.astype(np.float64)[:, None] - Ws)
    assert np.all(err <= sW.astype(np.float64)[:, None] * (0.5 + 1e-6))
    # compensated bias: b' - b equals z W^T (Eq. (g)) to fp32 rounding
    zw = W.astype(np.float64) @ z.astype(np.float64)
    np.testing.assert_allclose(bprime.astype(np.float64), zw + b.astype(np.float64),
                               rtol=2 ** -23, atol=1e-30)


def test_zero_weight_row_and_no_bias():
    W = np.zeros((2, 16), dtype=np.float16)
    W[1, 3] = 0.5
    z = np.full(16, 2.0, dtype=np.float32)
    s = np.full(16, 0.25, dtype=np.float32)
    Wq, sW, bprime = O.fold_weights(W, None, z, s, 8)
    assert sW[0] == 1.0 and not Wq[0].any()
    assert Wq[1, 3] == 127 and sW[1] == np.float32(0.125 / 127)
    assert bprime[0] == 0.0 and bprime[1] == 1.0


def test_non_finite_weights_rejected():
    W = np.ones((2, 16), dtype=np.float16)
    W[0, 0] = np.inf
    with pytest.raises(O.NonFinite):
        O.fold_weights(W, None, np.zeros(16, np.float32), np.ones(16, np.float32), 8)


# --------------------------------------------------------------------------
# Eq. (d) and Eq. (f) agree when nothing is rounded; Eq. (g) is exact too
# --------------------------------------------------------------------------
def test_internal_scaling_equals_folded_form_unrounded():
    r = np.random.default_rng(5)
    M, K, N = 4, 24, 6
    X = r.standard_normal((M, K))
    W = r.standard_normal((N, K))
    sX = r.uniform(0.1, 3.0, size=K)
    Ws = W * sX[None, :]
    sWs = np.abs(Ws).max(axis=1) / 127
    sWplain = np.abs(W).max(axis=1) / 127
    # left-hand side of Eq. (f): Eq. (d) with unrounded operands
    lhs = O.internal_scaling_fp64(X / sX[None, :], W / sWplain[:, None], sX, sWplain)
    # right-hand side of Eq. (f): no scale inside the sum
    rhs = sWs[None, :] * ((X / sX[None, :]) @ (Ws / sWs[:, None]).T)
    ref = X @ W.T
    np.testing.assert_allclose(lhs, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(rhs, ref, rtol=1e-12, atol=1e-12)


def test_symmetrized_fold_identity_fp64():
    wl = synth.WORKLOADS["opt125m_w8a8"]
    _, z, s, _ = O.calibrate(list(synth.calibration_batches(wl, 0)), 8)
    X = synth.activations(wl, 0, wl.M)
    W = synth.weight(wl, 0)
    b = synth.bias(wl, 0)
    ref = O.reference_fp64(X, W, b)
    fold = O.folded_fp64(X, W, b, z, s)
    np.testing.assert_allclose(fold, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


# --------------------------------------------------------------------------
# Quantizer (Eq. (a) made symmetric; Eq. (g))
# --------------------------------------------------------------------------
def test_quantizer_ties_to_even_and_clamps():
    x = np.array([[2.5, 3.5, -2.5, -0.5, 0.5, 1.5, 200.0, -200.0, 126.5, -127.5]],
                 dtype=np.float16)
    K = x.shape[1]
    z = np.zeros(K, np.float32)
    one = np.ones(K, np.float32)
    q = O.quantize_act(x, z, one, 8)
    expected = [round(float(v)) for v in x[0]]  # Python's round() is half-to-even
    expected = [max(-127, min(127, e)) for e in expected]
    np.testing.assert_array_equal(q[0], expected)
    q6 = O.quantize_act(x, z, one, 6)
    assert q6.max() == 31 and q6.min() == -31


def test_quantizer_identity_on_integer_grid():
    v = np.arange(-127, 128, dtype=np.float16)[None, :]
    K = v.shape[1]
    q = O.quantize_act(v, np.zeros(K, np.float32), np.ones(K, np.float32), 8)
    np.testing.assert_array_equal(q[0], np.arange(-127, 128))


def test_quantizer_matches_exact_rational_rounding():
    # the two float32 steps must match exact rational arithmetic rounded once
    # whenever the exact value is not within float32 rounding of a tie
    r = np.random.default_rng(3)
    x = r.normal(0, 4, size=(64, 32)).astype(np.float16)
    z = r.normal(0, 1, size=32).astype(np.float32)
    inv_s = r.uniform(5, 30, size=32).astype(np.float32)
    q = O.quantize_act(x, z, inv_s, 8)
    for i in range(0, 64, 7):
        for k in range(32):
            u = (Fraction(float(x[i, k])) - Fraction(float(z[k]))) * Fraction(float(inv_s[k]))
            frac = u - (u.numerator // u.denominator)
            if abs(frac - Fraction(1, 2)) < Fraction(1, 10 ** 4):
                continue
            ref = max(-127, min(127, round(u)))
            assert q[i, k] == ref


def test_per_tensor_special_case_reduces_to_eq_b():
    # all channels share one range and z = 0: per-channel quantization is
    # per-tensor quantization, and Y = s^X s^W sum_k Xt Wt (Eq. (b))
    r = np.random.default_rng(9)
    K, M, N = 32, 5, 4
    calib = r.uniform(-4, 4, size=(16, K)).astype(np.float16)
    calib[0, :] = -4.0
    calib[1, :] = 4.0
    _, z, s, inv_s = O.calibrate([calib], 8)
    assert np.all(z == 0) and np.all(s == s[0])
    W = np.clip(r.standard_normal((N, K)) * 0.02, -0.04, 0.04).astype(np.float16)
    W[:, 0] = 0.05  # every row has the same largest magnitude
    Wq, sW, bprime = O.fold_weights(W, None, z, s, 8)
    assert np.all(sW == sW[0]) and np.all(bprime == 0)
    X = r.uniform(-4, 4, size=(M, K)).astype(np.float16)
    Xt = np.array([[round(float(v) / float(s[0])) for v in row] for row in X.astype(np.float32)])
    Wt = np.array([[round(float(Fraction(float(w)) * Fraction(float(s[0])) / Fraction(float(sW[0]))))
                    for w in row] for row in W])
    np.testing.assert_array_equal(Wq, Wt)
    Y = O.epilogue_fp32(O.int_gemm(O.quantize_act(X, z, inv_s, 8), Wq), sW, bprime)
    eqb = float(sW[0]) * (Xt @ Wt.T)
    np.testing.assert_allclose(Y.astype(np.float64), eqb, rtol=2 ** -22)


# --------------------------------------------------------------------------
# Epilogue: int32 -> fp32 and fp32 -> fp16 conversions
# --------------------------------------------------------------------------
def test_epilogue_conversions_round_to_nearest_even():
    acc = np.array([[2 ** 24 + 1, 2 ** 24 + 3, -(2 ** 24 + 1), 7]], dtype=np.int32)
    sW = np.full(4, 2.0 ** -10, dtype=np.float32)
    y = O.epilogue_fp32(acc, sW, np.zeros(4, np.float32))
    np.testing.assert_array_equal(y[0], np.float32([2 ** 14, (2 ** 24 + 4) / 1024,
                                                    -(2 ** 14), 7 / 1024]))
    big = np.array([[65519, 65520, -65520, 1]], dtype=np.int32)
    Y = O.epilogue(big, np.ones(4, np.float32), np.float32([0, 0, 0, 2 ** -26]))
    assert Y[0, 0] == 65504 and np.isposinf(Y[0, 1]) and np.isneginf(Y[0, 2])
    assert Y[0, 3] == np.float16(1.0)


def test_epilogue_scales_by_output_channel():
    acc = np.array([[1, 1, 1], [2, 2, 2]], dtype=np.int32)
    Y = O.epilogue(acc, np.float32([1, 2, 4]), np.float32([0, 10, 100]))
    np.testing.assert_array_equal(Y, np.float16([[1, 12, 104], [2, 14, 108]]))


# --------------------------------------------------------------------------
# Approximation bound derived from Eq. (f)/(g)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("a_bits,w_bits", [(8, 8), (6, 6)])
def test_quantization_error_within_derived_bound(a_bits, w_bits):
    """For activations inside the calibrated range, |X_hat/s - q| <= 1/2 and
    |W_s/sW - Wq| <= 1/2, so
        |X W^T + b - (sW acc + b')| <= sW sum_k (|q|/2 + |Wq|/2 + 1/4)
    plus float32 rounding of b' and of the epilogue."""
    wl = synth.WORKLOADS["opt125m_w8a8"]
    batches = list(synth.calibration_batches(wl, 0))
    X = batches[0]  # inside the calibrated range by construction
    W = synth.weight(wl, 0)
    b = synth.bias(wl, 0)
    r = O.pipeline(X, W, b, batches, a_bits, w_bits)
    ref = O.reference_fp64(X, W, b)
    y = O.epilogue_fp32(r["acc"], r["sW"], r["bprime"]).astype(np.float64)
    q = np.abs(r["Xq"].astype(np.float64))
    wq = np.abs(r["Wq"].astype(np.float64))
    K = X.shape[1]
    bound = r["sW"].astype(np.float64)[None, :] * (q.sum(1)[:, None] / 2 + wq.sum(1)[None, :] / 2 + K / 4)
    slack = 4 * 2 ** -24 * (np.abs(y) + np.abs(r["bprime"]).astype(np.float64)[None, :]) + 1e-6
    err = np.abs(ref - y)
    assert np.all(err <= bound + slack)
    # and the error is far from vacuous: well under the bound on average
    assert err.mean() < 0.25 * bound.mean()


def test_symmetrization_lowers_error_on_offset_channels():
    """Sec. 3.2 / Table 6: symmetrization matters most at low bit-width on
    channels with offset ranges.  Without z the scale must cover max|X|."""
    wl = synth.WORKLOADS["opt13b_w6a6"]
    K = 256
    r = np.random.default_rng(1)
    off = r.uniform(-10, 10, size=K)
    x = (r.standard_normal((512, K)) + off[None, :]).astype(np.float16)
    W = (r.standard_normal((64, K)) * 0.02).astype(np.float16)
    _, z, s, inv_s = O.calibrate([x], 6)
    Wq, sW, bp = O.fold_weights(W, None, z, s, 6)
    y_sym = O.epilogue_fp32(O.int_gemm(O.quantize_act(x, z, inv_s, 6), Wq), sW, bp)
    # non-symmetrized: z = 0 and s = max|x| / qa
    z0 = np.zeros(K, np.float32)
    s0 = (np.abs(x.astype(np.float64)).max(0) / 31).astype(np.float32)
    inv0 = (1 / s0.astype(np.float64)).astype(np.float32)
    Wq0, sW0, bp0 = O.fold_weights(W, None, z0, s0, 6)
    y_non = O.epilogue_fp32(O.int_gemm(O.quantize_act(x, z0, inv0, 6), Wq0), sW0, bp0)
    ref = O.reference_fp64(x, W, None)
    e_sym = np.sqrt(np.mean((y_sym - ref) ** 2))
    e_non = np.sqrt(np.mean((y_non - ref) ** 2))
    assert e_sym < e_non
    del wl


# --------------------------------------------------------------------------
# Input generators
# --------------------------------------------------------------------------
def test_generators_are_deterministic_and_shaped():
    wl = synth.WORKLOADS["opt125m_w8a8"]
    a = synth.activations(wl, 0, 16)
    b = synth.activations(wl, 0, 16)
    assert a.dtype == np.float16 and a.shape == (16, 768)
    assert a.tobytes() == b.tobytes()
    c = next(synth.calibration_batches(wl, 0))
    assert c.tobytes() != a.tobytes()
    ch = synth.outlier_channels(wl, 0, 768)
    assert ch.size == 8
    # outlier channels are far larger and offset by +15 (the recipe)
    big = np.concatenate(list(synth.calibration_batches(wl, 0))).astype(np.float64)
    assert np.abs(big[:, ch]).mean() > 10 * np.abs(np.delete(big, ch, axis=1)).mean()
    assert abs(big[:, ch].mean() - 15) < 10
    W = synth.weight(wl, 0)
    assert W.shape == (768, 768) and abs(float(W.astype(np.float64).std()) - 0.02) < 1e-3

"""Pins for the oracle's per-token path (Eq. (c) and (h)): quantize_act_per_token,
fold_weights_per_token and epilogue_per_token, checked against what the paper
and plain arithmetic fix, never against a re-typed copy of the formula:

* a hand-worked example (3-bit codes, a tie, a zero row);
* each row's largest-magnitude value lands on +-qa, every code within range;
* with all rows sharing one scale the path is per-tensor quantization,
  Eq. (b): checked against numpy's matmul on integer codes;
* Eq. (h) with rounding disabled: s^W s^X (X/s^X)(W/s^W)^T + (b + z) plus the
  symmetrized residual X_res - z equals X W^T + b + X_res;
* the paper's Sec. 2.2 observation (i): on activations with outlier channels
  the per-token reconstruction error exceeds the per-channel one;
* the derived error bound of the whole per-token linear.

test_oracle_pt_mutations plants mistakes in the oracle and checks these fail.
"""
import numpy as np
import pytest

from oracle import ot_oracle as O


def test_hand_worked_example():
    X = np.array([[1, -4, 2, -2], [0, 0, 0, 0], [0.5, 0.25, -0.125, 1]], dtype=np.float16)
    q, s = O.quantize_act_per_token(X, 3)
    # row 0: s = 4/3, 1/s = 0.75 -> 0.75, -3, 1.5 (tie -> 2), -1.5 (tie -> -2)
    # row 1: zeros -> s = 1, codes 0;  row 2: s = 1/3, 1/s rounds to 3.0
    assert q.tolist() == [[1, -3, 2, -2], [0, 0, 0, 0], [2, 1, 0, 3]]
    assert s.tolist() == [np.float32(4 / 3), 1.0, np.float32(1 / 3)]
    W = np.array([[1.5, -3, 0, 0.75], [0, 0, 0, 0]], dtype=np.float16)
    Wq, sW, bp = O.fold_weights_per_token(W, np.array([0.5, -1], np.float16),
                                          np.array([0.25, 2], np.float32), 3)
    # row 0: sW = 3/3 = 1: 1.5 (tie -> 2), -3, 0, 0.75 -> 1; row 1: zero row, sW = 1
    # b' = b + z (Eq. (h)): 0.75, 1
    assert Wq.tolist() == [[2, -3, 0, 1], [0, 0, 0, 0]]
    assert sW.tolist() == [1.0, 1.0]
    assert bp.tolist() == [0.75, 1.0]
    acc = O.int_gemm(q, Wq)
    assert acc.tolist() == [[2 + 9 + 0 - 2, 0], [0, 0], [4 - 3 + 0 + 3, 0]]
    Y = O.epilogue_per_token(acc, s, sW, bp)
    # 9 * fp32(4/3) = 12.0000004 -> fp32 12 -> + 0.75 = 12.75 (exact in fp16)
    # 4 * fp32(1/3) = 1.3333334 -> + 0.75 = 2.0833335 -> fp16 2.083984375
    assert Y.astype(np.float64).tolist() == [[12.75, 1.0], [0.75, 1.0], [2.083984375, 1.0]]


@pytest.mark.parametrize("a_bits", [8, 6, 4])
def test_row_extremes_land_on_qmax(a_bits):
    r = np.random.default_rng(3)
    X = (r.standard_normal((32, 257)) * r.uniform(0.01, 100, (32, 1))).astype(np.float16)
    q, s = O.quantize_act_per_token(X, a_bits)
    qa = O.qmax(a_bits)
    i = np.abs(X.astype(np.float64)).argmax(axis=1)
    assert np.all(np.abs(q[np.arange(32), i]) == qa)
    assert np.all(np.abs(q.astype(int)) <= qa)
    # reconstruction within half a step, plus the fp32 roundings of 1/s and
    # of x * (1/s) (each 2^-24 relative, on |x/s| <= qa)
    err = np.abs(X.astype(np.float64) - q * s.astype(np.float64)[:, None])
    assert np.all(err <= s[:, None] * (0.5 + qa * 2.0 ** -22))


def test_equal_scales_reduce_to_per_tensor():
    """Rows that share one max |x| share one scale: Eq. (b)'s per-tensor form."""
    r = np.random.default_rng(4)
    X = r.uniform(-1, 1, (6, 96)).astype(np.float16)
    X[:, 0] = 2.0  # every row's max |x| is 2
    W = r.uniform(-1, 1, (5, 96)).astype(np.float16)
    q, s = O.quantize_act_per_token(X, 8)
    assert np.all(s == s[0])
    Wq, sW, bp = O.fold_weights_per_token(W, None, None, 8)
    acc = O.int_gemm(q, Wq)
    ref = q.astype(np.int64) @ Wq.astype(np.int64).T
    assert np.array_equal(acc, ref)
    Y = O.epilogue_per_token(acc, s, sW, bp).astype(np.float64)
    per_tensor = float(s[0]) * (ref * sW.astype(np.float64)[None, :])
    assert np.allclose(Y, per_tensor, rtol=2e-3, atol=1e-3)


def test_eq_h_identity_without_rounding():
    """Eq. (h) with unrounded quantizers: the per-token factorization plus the
    bias b + z and the symmetrized residual reproduces X W^T + b + X_res."""
    r = np.random.default_rng(8)
    M, K, N = 7, 40, 9
    X = r.normal(0, 1, (M, K))
    W = r.normal(0, 0.1, (N, K))
    b = r.normal(0, 0.1, N)
    z = r.normal(0, 1, N)
    Xres = r.normal(0, 1, (M, N))
    sX = np.abs(X).max(1) / 127.0
    sW = np.abs(W).max(1) / 127.0
    lhs = X @ W.T + b + Xres
    rhs = sW[None, :] * sX[:, None] * ((X / sX[:, None]) @ (W / sW[:, None]).T) + (b + z) \
        + (Xres - z)
    assert np.allclose(lhs, rhs, rtol=0, atol=1e-12)
    # the oracle's fold carries exactly b + z into b'
    Wh = W.astype(np.float16)
    _, _, bp = O.fold_weights_per_token(Wh, b.astype(np.float16), z.astype(np.float32), 8)
    assert np.array_equal(bp, (b.astype(np.float16).astype(np.float64)
                               + z.astype(np.float32)).astype(np.float32))


def test_outlier_channels_hurt_per_token_more_than_per_channel():
    """Sec. 2.2 (i): outlier channels dominate a token's range, so per-token
    codes reconstruct the normal channels worse than per-channel codes."""
    r = np.random.default_rng(10)
    X = r.standard_normal((64, 512))
    X[:, :5] *= 60
    X = X.astype(np.float16)
    q, s = O.quantize_act_per_token(X, 8)
    err_tok = np.abs(X.astype(np.float64) - q * s.astype(np.float64)[:, None])[:, 5:].mean()
    _, z, sc, inv = O.calibrate([X], 8)
    qc = O.quantize_act(X, z, inv, 8)
    err_ch = np.abs(X.astype(np.float64) - (qc * sc.astype(np.float64) + z))[:, 5:].mean()
    assert err_tok > 5 * err_ch


@pytest.mark.parametrize("a_bits,w_bits", [(8, 8), (6, 6), (8, 4)])
def test_per_token_linear_within_derived_bound(a_bits, w_bits):
    """|Y - (X W^T + b)| <= sX_m sW_n sum_k (|q|/2 + |Wq|/2 + 1/4) + fp16 rounding."""
    r = np.random.default_rng(a_bits * 10 + w_bits)
    M, K, N = 12, 200, 16
    X = r.normal(0, 1, (M, K)).astype(np.float16)
    W = r.normal(0, 0.05, (N, K)).astype(np.float16)
    b = r.normal(0, 0.1, N).astype(np.float16)
    q, sX = O.quantize_act_per_token(X, a_bits)
    Wq, sW, bp = O.fold_weights_per_token(W, b, None, w_bits)
    Y = O.epilogue_per_token(O.int_gemm(q, Wq), sX, sW, bp).astype(np.float64)
    ref = X.astype(np.float64) @ W.astype(np.float64).T + b.astype(np.float64)
    bound = (sX.astype(np.float64)[:, None] * sW.astype(np.float64)[None, :]
             * (np.abs(q).sum(1)[:, None] / 2 + np.abs(Wq).sum(1)[None, :] / 2 + K / 4))
    bound = bound * (1 + 1e-5) + np.abs(ref) * 2.0 ** -10 + 1e-3
    assert np.all(np.abs(Y - ref) <= bound)

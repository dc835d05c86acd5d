"""Pins for the oracle's asymmetric ("Int8") weights, Eq. (a) with a zero
point: fold_weights_asym and int_gemm_asym.

* a hand-worked 3-bit example (mixed-sign, all-positive and zero rows);
* zero is represented exactly, and every weight reconstructs to within half
  a step (the range always holds every value, so nothing clips);
* each row's minimum and maximum land on the end codes 0 and 2^b - 1;
* the integer sum against a Python triple loop on tiny shapes;
* on one-sided (skewed) rows the asymmetric quantizer reconstructs better
  than the symmetric Int8* one (the reason the paper offers both).
test_oracle_asym_mutations plants mistakes and checks these fail.
"""
import numpy as np
import pytest

from oracle import ot_oracle as O


def _ones(K):
    return np.ones(K, np.float32), np.zeros(K, np.float32)


def test_hand_worked_example():
    W = np.array([[-1, 0, 2.5, 6], [0.5, 1, 2, 3.5], [0, 0, 0, 0]], dtype=np.float16)
    s, z = _ones(4)
    Wq, sW, zW, bp = O.fold_weights_asym(W, None, z, s, 3)
    # row 0: lo -1, hi 6, sW = 7/7 = 1, zW = 1: codes rne(W)+1 = 0, 1, 3 (2.5 -> 2), 7
    # row 1: lo 0 (the range holds 0), hi 3.5, sW = 0.5, zW = 0: codes 1, 2, 4, 7
    # row 2: zero row, sW = 1, zW = 0; stored shifted by 4
    assert Wq.tolist() == [[-4, -3, -1, 3], [-3, -2, 0, 3], [-4, -4, -4, -4]]
    assert sW.tolist() == [1.0, 0.5, 1.0]
    assert zW.tolist() == [-3, -4, -4]
    Xq = np.array([[1, -2, 3, 0], [0, 0, 0, 1]], dtype=np.int8)
    acc = O.int_gemm_asym(Xq, Wq, zW)
    # c - zW: row 0 [-1, 0, 2, 6], row 1 [1, 2, 4, 7], row 2 zeros
    assert acc.tolist() == [[-1 + 0 + 6, 1 - 4 + 12, 0], [6, 7, 0]]


@pytest.mark.parametrize("w_bits", [8, 6, 4])
def test_zero_exact_and_half_step_reconstruction(w_bits):
    r = np.random.default_rng(w_bits)
    W = (r.standard_normal((40, 300)) * 0.05 + r.uniform(-0.1, 0.1, (40, 1))).astype(np.float16)
    W[:, :7] = 0.0
    s = r.uniform(0.2, 3.0, 300).astype(np.float32)
    z = np.zeros(300, np.float32)
    Wq, sW, zW, _ = O.fold_weights_asym(W, None, z, s, w_bits)
    deq = (Wq.astype(np.float64) - zW[:, None]) * sW.astype(np.float64)[:, None]
    Ws = W.astype(np.float64) * s.astype(np.float64)
    assert np.all(deq[:, :7] == 0.0)
    assert np.all(np.abs(deq - Ws) <= sW.astype(np.float64)[:, None] * (0.5 + 1e-6))
    L = (1 << w_bits) - 1
    c = Wq.astype(int) + (1 << (w_bits - 1))
    assert c.min() >= 0 and c.max() <= L
    # the row extremes take the end codes (within one where sW rounded up)
    rows_neg = Ws.min(1) < 0
    assert np.all(c[rows_neg].min(1) == 0)
    assert np.all(c.max(1) >= L - 1)


def test_integer_sum_against_triple_loop():
    r = np.random.default_rng(2)
    Xq = r.integers(-31, 32, (3, 5)).astype(np.int8)
    Wq = r.integers(-128, 128, (4, 5)).astype(np.int8)
    zW = r.integers(-128, 128, 4).astype(np.int32)
    acc = O.int_gemm_asym(Xq, Wq, zW)
    for m in range(3):
        for n in range(4):
            assert acc[m, n] == sum(int(Xq[m, k]) * (int(Wq[n, k]) - int(zW[n])) for k in range(5))


def test_asymmetric_beats_symmetric_on_one_sided_rows():
    r = np.random.default_rng(6)
    W = np.abs(r.standard_normal((32, 256)) * 0.05).astype(np.float16)  # all >= 0
    s, z = _ones(256)
    Wq, sW, zW, _ = O.fold_weights_asym(W, None, z, s, 6)
    deq_a = (Wq.astype(np.float64) - zW[:, None]) * sW.astype(np.float64)[:, None]
    Wq_s, sW_s, _ = O.fold_weights(W, None, z, s, 6)
    deq_s = Wq_s.astype(np.float64) * sW_s.astype(np.float64)[:, None]
    Wd = W.astype(np.float64)
    assert np.abs(deq_a - Wd).mean() < 0.6 * np.abs(deq_s - Wd).mean()

"""Pins for scales_from_minmax (scales from a calibration state, with and
without symmetrization): hand values, the codes it gives on the calibration
extremes, and agreement with calibrate where both apply."""
import numpy as np
import pytest

from oracle import ot_oracle as O


def test_hand_values():
    # channels: [-1, 3], [-2, 0], [5, 5], [-4, 2]
    mm = np.array([-1, -2, 5, -4, 3, 0, 5, 2], dtype=np.float32)
    z, s, inv = O.scales_from_minmax(mm, 3, True)      # qa = 3
    assert z.tolist() == [1.0, -1.0, 5.0, -1.0]
    assert s.tolist() == [np.float32(2 / 3), np.float32(1 / 3), 1.0, 1.0]
    z, s, inv = O.scales_from_minmax(mm, 3, False)
    assert z.tolist() == [0.0, 0.0, 0.0, 0.0]
    assert s.tolist() == [1.0, np.float32(2 / 3), np.float32(5 / 3), np.float32(4 / 3)]
    assert inv.tolist() == [1.0, 1.5, 0.6000000238418579, 0.75]


@pytest.mark.parametrize("a_bits", [8, 6, 4])
def test_extremes_map_to_qmax_and_nonsym_wastes_codes(a_bits):
    r = np.random.default_rng(a_bits)
    X = (r.standard_normal((512, 64)) + r.uniform(-8, 8, 64)).astype(np.float16)
    mm, _, _, _ = O.calibrate([X], a_bits)
    qa = O.qmax(a_bits)
    zs, ss, invs = O.scales_from_minmax(mm, a_bits, True)
    q = O.quantize_act(X, zs, invs, a_bits)
    assert np.all(q.max(0) == qa) and np.all(q.min(0) == -qa)
    zn, sn, invn = O.scales_from_minmax(mm, a_bits, False)
    qn = O.quantize_act(X, zn, invn, a_bits)
    # the side with the larger magnitude reaches qa; offset channels leave
    # most of the other side unused
    assert np.all(np.maximum(qn.max(0), -qn.min(0).astype(int)) == qa)
    used_sym = (q.max(0).astype(int) - q.min(0)).mean()
    used_non = (qn.max(0).astype(int) - qn.min(0)).mean()
    assert used_non < 0.8 * used_sym
    # reconstruction error: symmetrized is smaller on offset channels
    err_s = np.abs(X.astype(np.float64) - (q * ss.astype(np.float64) + zs)).mean()
    err_n = np.abs(X.astype(np.float64) - qn * sn.astype(np.float64)).mean()
    assert err_s < err_n


@pytest.mark.parametrize("a_bits", [8, 6, 3])
def test_symmetrized_scales_equal_calibrate(a_bits):
    r = np.random.default_rng(11)
    batches = [(r.standard_normal((33, 40)) * 3 + 1).astype(np.float16) for _ in range(3)]
    mm, z, s, inv = O.calibrate(batches, a_bits)
    z2, s2, inv2 = O.scales_from_minmax(mm, a_bits, True)
    for a, b in ((z, z2), (s, s2), (inv, inv2)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))

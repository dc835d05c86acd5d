"""Plants mistakes in scales_from_minmax (on the CPU) and checks that the
pins in test_oracle_sweep_pins catch each one."""
import numpy as np
import pytest

from oracle import ot_oracle as O
from tests import test_oracle_sweep_pins as P


def _pins_pass():
    try:
        P.test_hand_values()
        for ab in (8, 6, 4):
            P.test_extremes_map_to_qmax_and_nonsym_wastes_codes(ab)
        for ab in (8, 6, 3):
            P.test_symmetrized_scales_equal_calibrate(ab)
    except (AssertionError, ValueError, IndexError):
        return False
    return True


def _mut(nonsym_abs=True, half=2.0, shift_sign=1.0):
    def scales_from_minmax(minmax, a_bits, symmetrize=True):
        qa = O.qmax(a_bits)
        mm = np.asarray(minmax, np.float32).astype(np.float64)
        K = mm.size // 2
        lo, hi = mm[:K], mm[K:]
        if symmetrize:
            z = ((hi + shift_sign * lo) / 2).astype(np.float32)
            s = (((hi - lo) / half) / qa).astype(np.float32)
        else:
            z = np.zeros(K, np.float32)
            m = np.maximum(np.abs(lo), np.abs(hi)) if nonsym_abs else np.maximum(lo, hi)
            s = (m / qa).astype(np.float32)
        s[s == 0] = 1
        return z, s, (1 / s.astype(np.float64)).astype(np.float32)
    return scales_from_minmax


MUTANTS = {"nonsym_without_abs": _mut(nonsym_abs=False), "full_range_scale": _mut(half=1.0),
           "shift_uses_difference": _mut(shift_sign=-1.0)}


def test_unmutated_oracle_passes_sweep_pins():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_sweep_pins_catch_mutant(name, monkeypatch):
    monkeypatch.setattr(O, "scales_from_minmax", MUTANTS[name])
    assert not _pins_pass(), f"mutant {name} slipped through"

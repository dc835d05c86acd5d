"""Plants mistakes in the oracle's asymmetric weights (on the CPU) and checks
that the pins in test_oracle_asym_pins catch each one."""
import numpy as np
import pytest

from oracle import ot_oracle as O
from tests import test_oracle_asym_pins as P


def _pins_pass():
    try:
        P.test_hand_worked_example()
        for wb in (8, 6, 4):
            P.test_zero_exact_and_half_step_reconstruction(wb)
        P.test_integer_sum_against_triple_loop()
        P.test_asymmetric_beats_symmetric_on_one_sided_rows()
    except (AssertionError, ValueError, IndexError):
        return False
    return True


def _fold(levels_offset=0, include_zero=True, zp_sign=1.0):
    def fold_weights_asym(W, b, z, s, w_bits):
        L = (1 << w_bits) - 1 + levels_offset
        half = 1 << (w_bits - 1)
        W64 = np.asarray(W).astype(np.float64)
        Ws = W64 * np.asarray(s, np.float32).astype(np.float64)[None, :]
        lo, hi = Ws.min(1), Ws.max(1)
        if include_zero:
            lo, hi = np.minimum(lo, 0), np.maximum(hi, 0)
        sW = ((hi - lo) / L).astype(np.float32)
        sW[sW == 0] = 1
        zW = np.clip(np.rint(zp_sign * -lo / sW.astype(np.float64)), 0, (1 << w_bits) - 1)
        c = np.clip(np.rint(Ws / sW.astype(np.float64)[:, None]) + zW[:, None], 0,
                    (1 << w_bits) - 1)
        bp = (W64 @ np.asarray(z, np.float64) + (0 if b is None else np.asarray(b, np.float64)))
        return (c - half).astype(np.int8), sW, (zW - half).astype(np.int32), bp.astype(np.float32)
    return fold_weights_asym


def _gemm_no_zero_point(Xq, Wq, zWq):
    return (np.asarray(Xq, np.float64) @ np.asarray(Wq, np.float64).T).astype(np.int32)


MUTANTS = {
    "levels_2_to_the_b": ("fold_weights_asym", _fold(levels_offset=1)),
    "range_without_zero": ("fold_weights_asym", _fold(include_zero=False)),
    "zero_point_sign": ("fold_weights_asym", _fold(zp_sign=-1.0)),
    "gemm_ignores_zero_point": ("int_gemm_asym", _gemm_no_zero_point),
}


def test_unmutated_oracle_passes_asym_pins():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_asym_pins_catch_mutant(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(O, attr, fn)
    assert not _pins_pass(), f"mutant {name} slipped through the asymmetric-weight pins"

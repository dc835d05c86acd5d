"""Plants plausible mistakes in the oracle (on the CPU) and checks that the
pins in test_oracle_pins catch every one of them.

Each mutant replaces one oracle function with a subtly wrong copy (a dropped
term, a wrong sign, a wrong axis, a different rounding); the hand-worked
example and the rounding-free identity must then fail.
"""
import numpy as np
import pytest

from oracle import ot_oracle as O
from tests import test_oracle_pins as P


def _pins_pass():
    try:
        P.test_hand_worked_example_every_stage()
        for ab, wb in [(8, 8), (6, 6)]:
            P.test_rounding_free_fold_reproduces_linear_exactly(ab, wb)
        P.test_quantizer_ties_to_even_and_clamps()
        P.test_epilogue_scales_by_output_channel()
    except (AssertionError, ValueError, IndexError):
        return False
    return True


def _calib_factory(z_sign=1.0, half_div=2.0):
    def calibrate(batches, a_bits):
        qa = O.qmax(a_bits)
        x = np.concatenate([np.asarray(b).astype(np.float64) for b in batches])
        lo, hi = x.min(0), x.max(0)
        z = ((hi + z_sign * lo) / 2.0).astype(np.float32)
        s = (((hi - lo) / half_div) / qa).astype(np.float32)
        s[s == 0] = 1
        return (np.concatenate([lo, hi]).astype(np.float32), z, s,
                (1 / s.astype(np.float64)).astype(np.float32))
    return calibrate


def _fold_factory(bias_from_folded=False, drop_bias=False, scale_round="rint"):
    def fold_weights(W, b, z, s, w_bits):
        qw = O.qmax(w_bits)
        W64 = np.asarray(W).astype(np.float64)
        Ws = W64 * np.asarray(s, np.float64)[None, :]
        sW = (np.abs(Ws).max(1) / qw).astype(np.float32)
        sW[sW == 0] = 1
        r = Ws / sW.astype(np.float64)[:, None]
        r = np.floor(r + 0.5) if scale_round == "half_up" else np.rint(r)
        Wq = np.clip(r, -qw, qw).astype(np.int8)
        src = Ws if bias_from_folded else W64
        bp = src @ np.asarray(z, np.float64)
        if not drop_bias and b is not None:
            bp = bp + np.asarray(b).astype(np.float64)
        return Wq, sW, bp.astype(np.float32)
    return fold_weights


def _quant_factory(z_sign=-1.0, rounding="rint"):
    def quantize_act(X, z, inv_s, a_bits):
        qa = O.qmax(a_bits)
        t = np.asarray(X).astype(np.float32) + np.float32(z_sign) * np.asarray(z, np.float32)[None, :]
        u = t * np.asarray(inv_s, np.float32)[None, :]
        r = np.floor(u + np.float32(0.5)) if rounding == "half_up" else np.rint(u)
        return np.clip(r, -qa, qa).astype(np.int8)
    return quantize_act


def _epi_factory(axis_rows=False, drop_bias=False):
    def epilogue_fp32(acc, sW, bprime):
        v = np.asarray(acc, np.int32).astype(np.float32)
        sW = np.asarray(sW, np.float32)
        if axis_rows:
            p = v * np.resize(sW, v.shape[0])[:, None]
        else:
            p = v * sW[None, :]
        return p if drop_bias else p + np.asarray(bprime, np.float32)[None, :]
    return epilogue_fp32


def _gemm_wrong_operand(Xq, Wq):
    # uses Wq's rows as if they were columns of a [K, N] matrix
    K = Xq.shape[1]
    flat = np.asarray(Wq).reshape(-1)[: K * Wq.shape[0]].reshape(K, Wq.shape[0])
    return (Xq.astype(np.float64) @ flat.astype(np.float64)).astype(np.int32)


MUTANTS = {
    "z_uses_difference": ("calibrate", _calib_factory(z_sign=-1.0)),
    "scale_missing_half": ("calibrate", _calib_factory(half_div=1.0)),
    "bias_from_folded_weight": ("fold_weights", _fold_factory(bias_from_folded=True)),
    "bias_dropped_in_fold": ("fold_weights", _fold_factory(drop_bias=True)),
    "weight_round_half_up": ("fold_weights", _fold_factory(scale_round="half_up")),
    "shift_added_not_subtracted": ("quantize_act", _quant_factory(z_sign=1.0)),
    "act_round_half_up": ("quantize_act", _quant_factory(rounding="half_up")),
    "gemm_wrong_operand_layout": ("int_gemm", _gemm_wrong_operand),
    "scale_on_token_axis": ("epilogue_fp32", _epi_factory(axis_rows=True)),
    "bias_dropped_in_epilogue": ("epilogue_fp32", _epi_factory(drop_bias=True)),
}


def test_unmutated_oracle_passes_pins():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    fn_name, fn = MUTANTS[name]
    monkeypatch.setattr(O, fn_name, fn)
    assert not _pins_pass(), f"mutant {name} survived the pins"

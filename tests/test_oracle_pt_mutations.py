"""Plants plausible mistakes in the oracle's per-token path (on the CPU) and
checks that the pins in test_oracle_pt_pins catch each one."""
import numpy as np
import pytest

from oracle import ot_oracle as O
from tests import test_oracle_pt_pins as P


def _pins_pass():
    try:
        P.test_hand_worked_example()
        for ab in (8, 6, 4):
            P.test_row_extremes_land_on_qmax(ab)
        P.test_equal_scales_reduce_to_per_tensor()
        P.test_eq_h_identity_without_rounding()
        P.test_outlier_channels_hurt_per_token_more_than_per_channel()
        for ab, wb in ((8, 8), (6, 6), (8, 4)):
            P.test_per_token_linear_within_derived_bound(ab, wb)
    except (AssertionError, ValueError, IndexError):
        return False
    return True


def _quant(axis=1, divisor_offset=0, rounding="rint"):
    def quantize_act_per_token(X, a_bits):
        qa = O.qmax(a_bits)
        x = np.asarray(X).astype(np.float64)
        mx = np.abs(x).max(axis=axis)
        s = (mx / float(qa + divisor_offset)).astype(np.float32)
        s[s == 0] = 1
        inv = (1 / s.astype(np.float64)).astype(np.float32)
        u = np.asarray(X).astype(np.float32) * (inv[:, None] if axis == 1 else inv[None, :])
        r = np.floor(u + 0.5) if rounding == "half_up" else np.rint(u)
        q = np.clip(r, -qa, qa).astype(np.int8)
        if axis != 1:  # per-channel scales reported as if per token
            s = np.resize(s, x.shape[0])
        return q, s
    return quantize_act_per_token


def _fold(z_sign=1.0, use_bias=True):
    def fold_weights_per_token(W, b, zres, w_bits):
        qw = O.qmax(w_bits)
        W64 = np.asarray(W).astype(np.float64)
        sW = (np.abs(W64).max(1) / qw).astype(np.float32)
        sW[sW == 0] = 1
        Wq = np.clip(np.rint(W64 / sW.astype(np.float64)[:, None]), -qw, qw).astype(np.int8)
        bp = np.zeros(W64.shape[0])
        if use_bias and b is not None:
            bp = bp + np.asarray(b).astype(np.float64)
        if zres is not None:
            bp = bp + z_sign * np.asarray(zres, np.float32).astype(np.float64)
        return Wq, sW, bp.astype(np.float32)
    return fold_weights_per_token


def _epi(swap=False, drop_token_scale=False):
    def epilogue_per_token(acc, sX, sW, bprime):
        a = np.asarray(acc, np.int64).astype(np.float32)
        sx = np.asarray(sX, np.float32)
        sw = np.asarray(sW, np.float32)
        if swap:  # token scale indexed by channel and vice versa
            sx, sw = np.resize(sw, sx.shape), np.resize(sx, sw.shape)
        t = a if drop_token_scale else a * sx[:, None]
        y = t * sw[None, :] + np.asarray(bprime, np.float32)[None, :]
        return y.astype(np.float16)
    return epilogue_per_token


MUTANTS = {
    "scale_per_channel_not_per_token": ("quantize_act_per_token", _quant(axis=0)),
    "scale_divides_by_qa_plus_1": ("quantize_act_per_token", _quant(divisor_offset=1)),
    "round_half_up": ("quantize_act_per_token", _quant(rounding="half_up")),
    "residual_shift_subtracted": ("fold_weights_per_token", _fold(z_sign=-1.0)),
    "bias_dropped": ("fold_weights_per_token", _fold(use_bias=False)),
    "scales_swapped": ("epilogue_per_token", _epi(swap=True)),
    "token_scale_dropped": ("epilogue_per_token", _epi(drop_token_scale=True)),
}


def test_unmutated_oracle_passes_pt_pins():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pt_pins_catch_mutant(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(O, attr, fn)
    assert not _pins_pass(), f"mutant {name} slipped through the per-token pins"

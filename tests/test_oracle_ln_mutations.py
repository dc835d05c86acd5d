"""Plants plausible mistakes in the oracle's LayerNorm-fused quantizer (on
the CPU) and checks that the pins in test_oracle_ln_pins catch each one."""
import math

import numpy as np
import pytest

from oracle import ot_oracle as O
from tests import test_oracle_ln_pins as P


def _pins_pass():
    try:
        P.test_stats_closed_form_rows()
        for sc in (1e-6, 1.0, 300.0, 5e3):
            P.test_stats_match_numpy_float64(sc)
        P.test_hand_worked_example_every_step()
        for ab in (8, 6):
            P.test_codes_match_textbook_layernorm_then_quantize(ab)
        P.test_power_of_two_scaling_leaves_codes_unchanged()
        P.test_constant_row_quantizes_the_shifted_bias()
    except (AssertionError, ValueError, IndexError):
        return False
    return True


def _stats(divisor_minus=0, drop_square_of_mean=False):
    def layernorm_stats(H):
        h = np.asarray(H).astype(np.float64)
        K = h.shape[1]
        mean = h.mean(1)
        if drop_square_of_mean:
            var = (h * h).mean(1)
        else:
            var = ((h - mean[:, None]) ** 2).sum(1) / (K - divisor_minus)
        return mean, var
    return layernorm_stats


def _lnq(c_sign=-1.0, use_gamma=True, use_eps=True, use_mean=True, rstd_op="rsqrt"):
    def ln_quantize_act(H, gamma, beta, eps, z, inv_s, a_bits):
        qa = O.qmax(a_bits)
        mean, var = O.layernorm_stats(H)
        e = float(np.float32(eps)) if use_eps else 0.0
        if rstd_op == "rsqrt":
            rstd = np.array([1.0 / math.sqrt(v + e) for v in var])
        else:  # forgot the square root
            rstd = np.array([1.0 / (v + e) if v + e else np.inf for v in var])
        mu32 = mean.astype(np.float32)[:, None] if use_mean else np.float32(0)
        d = np.asarray(H).astype(np.float32) - mu32
        n = d * rstd.astype(np.float32)[:, None]
        g = n * np.asarray(gamma).astype(np.float32)[None, :] if use_gamma else n
        c = np.asarray(beta).astype(np.float32) + np.float32(c_sign) * np.asarray(z, np.float32)
        u = (g + c[None, :]) * np.asarray(inv_s, np.float32)[None, :]
        return np.clip(np.rint(u), -qa, qa).astype(np.int8)
    return ln_quantize_act


MUTANTS = {
    "variance_divisor_K_minus_1": ("layernorm_stats", _stats(divisor_minus=1)),
    "variance_without_mean": ("layernorm_stats", _stats(drop_square_of_mean=True)),
    "shift_added_not_subtracted": ("ln_quantize_act", _lnq(c_sign=1.0)),
    "gamma_ignored": ("ln_quantize_act", _lnq(use_gamma=False)),
    "eps_ignored": ("ln_quantize_act", _lnq(use_eps=False)),
    "mean_not_subtracted": ("ln_quantize_act", _lnq(use_mean=False)),
    "rstd_without_sqrt": ("ln_quantize_act", _lnq(rstd_op="recip")),
}


def test_unmutated_oracle_passes_ln_pins():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_ln_pins_catch_mutant(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(O, attr, fn)
    assert not _pins_pass(), f"mutant {name} slipped through the LayerNorm pins"

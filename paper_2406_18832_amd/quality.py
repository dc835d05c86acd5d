"""Output error of the quantized linear against float64, on the synthetic
workloads: a symmetrization ablation and bit-width sweep standing in for the
paper's Table 6 (with and without symmetrization, Sec. 4.4) and Table 10
(W8A6, W6A6, W8A4, W4A4), plus the per-token path of Eq. (c) as the
baseline the paper argues against (Sec. 2.2).

The paper measures perplexity on checkpoints and datasets that are not used
here; this measures the error the method introduces in one linear, which is
what those numbers follow from.  Every step runs through libot: one
calibration pass (ot_calibrate) gives the minmax state, ot_scales_from_minmax
derives each configuration's z and s from it, then ot_fold_weights,
ot_quantize_act and ot_qlinear (or the per-token entry points).  The
reference is X W^T + b in float64 (torch, on the GPU).
"""
from __future__ import annotations

import torch

from . import ot, synth

# (label, a_bits, w_bits, path): path "channel" is OutlierTune's per-channel
# path, "channel-nosym" the same without symmetrization, "token" Eq. (c)
CONFIGS = [
    ("W8A8", 8, 8, "channel"), ("W8A8 no-sym", 8, 8, "channel-nosym"),
    ("W8A6", 6, 8, "channel"), ("W8A6 no-sym", 6, 8, "channel-nosym"),
    ("W6A6", 6, 6, "channel"), ("W6A6 no-sym", 6, 6, "channel-nosym"),
    ("W8A4", 4, 8, "channel"), ("W8A4 no-sym", 4, 8, "channel-nosym"),
    ("W4A4", 4, 4, "channel"), ("W4A4 no-sym", 4, 4, "channel-nosym"),
    ("W8A8 per-token", 8, 8, "token"), ("W6A6 per-token", 6, 6, "token"),
]


def layer_inputs(wl, li, rows, calib_rows, calib_batches, device="cuda"):
    """Device tensors of one layer: X [rows, K], W, b, and the calibration
    minmax state of ot_calibrate over the seeded calibration batches."""
    X = torch.from_numpy(synth.activations(wl, li, rows)).to(device)
    W = torch.from_numpy(synth.weight(wl, li)).to(device)
    b = torch.from_numpy(synth.bias(wl, li)).to(device)
    minmax, _, _, _ = ot.calibrate(synth.calibration_batches(wl, li, calib_rows, calib_batches),
                                   8, device)
    return X, W, b, minmax


def run_config(X, W, b, minmax, a_bits, w_bits, path):
    """The quantized linear's fp16 output for one configuration."""
    if path == "token":
        Xq, sX = ot.quantize_act_per_token(X, a_bits)
        Wq, sW, bp = ot.fold_weights_per_token(W, b, None, w_bits)
        return ot.qlinear_per_token(Xq, Wq, sX, sW, bp, a_bits, w_bits)
    z, s, inv_s = ot.scales_from_minmax(minmax, a_bits, path == "channel")
    Wq, sW, bp = ot.fold_weights(W, b, w_bits, z, s)
    Xq = ot.quantize_act(X, a_bits, z, inv_s)
    return ot.qlinear(Xq, Wq, sW, bp, a_bits, w_bits)


def errors(Y, ref):
    """Relative Frobenius error, mean and max absolute error (float64)."""
    e = Y.double() - ref
    return dict(rel_fro=float(e.norm() / ref.norm()), mean_abs=float(e.abs().mean()),
                max_abs=float(e.abs().max()))


def sweep(workloads=("opt6.7b_w8a8", "opt13b_w6a6", "opt66b_w8a8"), rows=256, calib_rows=None,
          calib_batches=None, configs=CONFIGS, device="cuda", log=None):
    """Errors of every configuration on every linear of the given workloads
    (calibration: the workload's own batches unless given).  Returns a list
    of dicts (workload, layer, config, a_bits, w_bits, path, rel_fro,
    mean_abs, max_abs)."""
    out = []
    for name in workloads:
        wl = synth.WORKLOADS[name]
        for li, lay in enumerate(wl.layers):
            X, W, b, minmax = layer_inputs(wl, li, rows, calib_rows, calib_batches, device)
            ref = torch.matmul(X.double(), W.double().t()) + b.double()
            for label, a_bits, w_bits, path in configs:
                Y = run_config(X, W, b, minmax, a_bits, w_bits, path)
                rec = dict(workload=name, layer=lay.name, config=label, a_bits=a_bits,
                           w_bits=w_bits, path=path, **errors(Y, ref))
                out.append(rec)
                if log:
                    log(f"quality {name}/{lay.name} {label}: rel {rec['rel_fro']:.3e}")
            del X, W, b, minmax, ref
    return out

"""The symmetrization ablation and bit-width sweep (paper_2406_18832_amd.quality)
on the GPU: every configuration's output equals the oracle's for the same
configuration, and the paper's qualitative findings hold on the synthetic
workloads (Sec. 4.4 / Table 6: without symmetrization low bit-widths break
down where channels are offset; Table 10: the error grows as bits drop).
The per-token rows are measured but carry no claim: on these layers the
per-channel path's error is dominated by quantizing the folded weights
(the paper's Table 10 finding), which puts it level with per-token at W8A8."""
import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import quality, synth
from tests._tol import assert_fp16_close

pytestmark = pytest.mark.gpu


def case(msg):
    print(f"[case] {msg}", flush=True)


def _oracle_config(X, W, b, batches, a_bits, w_bits, path):
    if path == "token":
        q, sX = O.quantize_act_per_token(X, a_bits)
        Wq, sW, bp = O.fold_weights_per_token(W, b, None, w_bits)
        return O.epilogue_per_token(O.int_gemm(q, Wq), sX, sW, bp)
    mm, _, _, _ = O.calibrate(batches, 8)
    z, s, inv = O.scales_from_minmax(mm, a_bits, path == "channel")
    Wq, sW, bp = O.fold_weights(W, b, z, s, w_bits)
    q = O.quantize_act(X, z, inv, a_bits)
    return O.epilogue(O.int_gemm(q, Wq), sW, bp)


@pytest.mark.parametrize("label,a_bits,w_bits,path", quality.CONFIGS)
def test_every_configuration_matches_the_oracle(label, a_bits, w_bits, path):
    wl = synth.WORKLOADS["opt125m_w8a8"]
    case(f"quality parity opt125m {label}")
    X, W, b, minmax = quality.layer_inputs(wl, 0, 16, 16, 4)
    Y = quality.run_config(X, W, b, minmax, a_bits, w_bits, path)
    batches = list(synth.calibration_batches(wl, 0, 16, 4))
    ref = _oracle_config(X.cpu().numpy(), W.cpu().numpy(), b.cpu().numpy(), batches, a_bits,
                         w_bits, path)
    assert_fp16_close(Y.cpu().numpy(), ref)


def _rel(records, layer, label):
    (r,) = [x for x in records if x["layer"] == layer and x["config"] == label]
    return r["rel_fro"]


def test_paper_findings_hold_on_synthetic_workloads():
    case("quality sweep opt13b + opt6.7b")
    recs = quality.sweep(workloads=("opt13b_w6a6", "opt6.7b_w8a8"), rows=128, calib_rows=256,
                         calib_batches=2)
    by = {}
    for r in recs:
        by.setdefault(r["workload"], []).append(r)
    for name, rs in by.items():
        for layer in ("qkv", "fc1"):
            e = {c[0]: _rel(rs, layer, c[0]) for c in quality.CONFIGS}
            # Table 10: fewer bits, larger error
            assert e["W8A8"] < e["W8A6"] < e["W8A4"] < e["W4A4"], (name, layer, e)
            assert e["W8A6"] < e["W6A6"], (name, layer, e)
    # Table 6 / Sec. 4.4: symmetrization matters where channels are offset
    # (the OPT-13B recipe shifts every channel), and is neutral where they
    # are centred (the OPT-6.7B recipe's activations are zero-mean)
    for layer in ("qkv", "fc1"):
        e = {c[0]: _rel(by["opt13b_w6a6"], layer, c[0]) for c in quality.CONFIGS}
        for bits in ("W8A8", "W8A6", "W6A6", "W8A4", "W4A4"):
            assert e[bits] < e[bits + " no-sym"], (layer, bits, e)
        e = {c[0]: _rel(by["opt6.7b_w8a8"], layer, c[0]) for c in quality.CONFIGS}
        for bits in ("W8A8", "W6A6"):
            assert abs(e[bits] - e[bits + " no-sym"]) < 0.15 * e[bits], (layer, bits, e)
    # the offset-heavy OPT-13B recipe: without symmetrization W6A6 and W4A4
    # break down (Table 6's Int6 rows), with it they degrade gradually
    e13 = {c[0]: _rel(by["opt13b_w6a6"], "qkv", c[0]) for c in quality.CONFIGS}
    assert e13["W6A6 no-sym"] > 2 * e13["W6A6"], e13
    assert e13["W4A4 no-sym"] > 3 * e13["W4A4"], e13

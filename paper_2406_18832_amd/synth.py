"""Seeded synthetic workloads shaped like the OPT linears the paper quantizes.

This module only draws numbers.  It holds none of the quantization method's
arithmetic (no scales, no shifts, no rounding to codes), so both the HIP path
and the CPU oracle may consume its output: they then see the same fp16 bytes.

The paper's data (Pile calibration sentences, Sec. 4.1 and App. A; OPT
checkpoints) is not used.  Each workload instead reproduces the property the
method exists for (Sec. 1, Sec. 2.2 "Limitations of different quantization
dimensions"): a few fixed activation channels carry structured outliers that
are far larger, and in places asymmetric, compared with the rest.

Seeding: every array is drawn from
``numpy.random.default_rng([20240626, cfg_index, layer_index, role, idx])``
with ``role`` one of the ``ROLE_*`` constants below, so any array can be
regenerated on its own, on any machine, byte for byte.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 20240626

ROLE_EVAL_X = 0      # the activations the timed linear consumes
ROLE_CALIB_X = 1     # calibration batch ``idx``
ROLE_WEIGHT = 2
ROLE_BIAS = 3
ROLE_OUTLIER_SET = 4  # which channels are outliers (fixed per layer)
ROLE_OFFSETS = 5      # per-channel mean offsets (fixed per layer)
ROLE_LN_INPUT = 6     # LayerNorm input rows: idx 0 evaluated, 1.. calibration
ROLE_LN_PARAMS = 7    # LayerNorm gain and bias, and the input's channel moments


@dataclass(frozen=True)
class Layer:
    name: str
    K: int  # in-features
    N: int  # out-features


@dataclass(frozen=True)
class Workload:
    """One synthetic quantized-linear workload.

    ``dist`` names the activation recipe implemented in :func:`activations`.
    """
    index: int
    name: str
    M: int
    layers: tuple
    a_bits: int
    w_bits: int
    dist: str
    outlier_frac: float
    n_outliers_fixed: int  # >0 overrides outlier_frac
    w_std: float
    b_std: float
    calib_batches: int
    calib_rows: int
    decode_M: tuple = field(default=())

    def layer(self, name: str) -> Layer:
        for lay in self.layers:
            if lay.name == name:
                return lay
        raise KeyError(name)


def _opt_block(hidden: int, ffn: int) -> tuple:
    return (Layer("qkv", hidden, 3 * hidden), Layer("out", hidden, hidden),
            Layer("fc1", hidden, ffn), Layer("fc2", ffn, hidden))


WORKLOADS = {
    # OPT-125m-shaped single linear, W8A8, 16 tokens; small enough for the
    # oracle to finish in seconds.
    "opt125m_w8a8": Workload(
        index=0, name="opt125m_w8a8", M=16, layers=(Layer("fc", 768, 768),),
        a_bits=8, w_bits=8, dist="normal_fixed8", outlier_frac=0.0,
        n_outliers_fixed=8, w_std=0.02, b_std=0.02, calib_batches=4,
        calib_rows=16),
    # OPT-6.7B decoder block linears, W8A8, 4x512 tokens; fc2's input is the
    # ReLU of fc1's output (non-negative, so strongly asymmetric).
    "opt6.7b_w8a8": Workload(
        index=1, name="opt6.7b_w8a8", M=2048, layers=_opt_block(4096, 16384),
        a_bits=8, w_bits=8, dist="normal_x60", outlier_frac=0.005,
        n_outliers_fixed=0, w_std=0.02, b_std=0.02, calib_batches=8,
        calib_rows=2048),
    # OPT-13B block, W6A6 (codes in [-31, 31] held in int8), 4096 tokens,
    # every channel carries a mean offset.
    "opt13b_w6a6": Workload(
        index=2, name="opt13b_w6a6", M=4096, layers=_opt_block(5120, 20480),
        a_bits=6, w_bits=6, dist="offset_x50", outlier_frac=0.01,
        n_outliers_fixed=0, w_std=0.02, b_std=0.02, calib_batches=8,
        calib_rows=2048),
    # OPT-30B block in the decode regime (a handful of tokens per step).
    "opt30b_decode_w8a8": Workload(
        index=3, name="opt30b_decode_w8a8", M=64, layers=_opt_block(7168, 28672),
        a_bits=8, w_bits=8, dist="normal_x60", outlier_frac=0.005,
        n_outliers_fixed=0, w_std=0.02, b_std=0.02, calib_batches=8,
        calib_rows=2048, decode_M=(1, 8, 32, 64)),
    # OPT-66B block, W8A8, 8192-token prefill, heavy-tailed activations.
    "opt66b_w8a8": Workload(
        index=4, name="opt66b_w8a8", M=8192, layers=_opt_block(9216, 36864),
        a_bits=8, w_bits=8, dist="laplace_x100", outlier_frac=0.01,
        n_outliers_fixed=0, w_std=0.015, b_std=0.015, calib_batches=8,
        calib_rows=2048),
}


def rng(wl: Workload, layer_index: int, role: int, idx: int = 0) -> np.random.Generator:
    return np.random.default_rng([SEED_BASE, wl.index, layer_index, role, idx])


def outlier_channels(wl: Workload, layer_index: int, K: int) -> np.ndarray:
    """Sorted indices of the fixed outlier channels of one layer's input."""
    n = wl.n_outliers_fixed if wl.n_outliers_fixed > 0 else int(round(wl.outlier_frac * K))
    n = min(n, K)
    g = rng(wl, layer_index, ROLE_OUTLIER_SET)
    return np.sort(g.choice(K, size=n, replace=False)).astype(np.int64)


def channel_offsets(wl: Workload, layer_index: int, K: int) -> np.ndarray:
    """Per-channel mean offsets (float64 [K]); zero where the recipe has none."""
    g = rng(wl, layer_index, ROLE_OFFSETS)
    if wl.dist == "offset_x50":
        return g.uniform(-10.0, 10.0, size=K)
    if wl.dist == "laplace_x100":
        off = np.zeros(K)
        ch = outlier_channels(wl, layer_index, K)
        off[ch] = g.uniform(-20.0, 20.0, size=ch.size)
        return off
    if wl.dist == "normal_fixed8":
        off = np.zeros(K)
        off[outlier_channels(wl, layer_index, K)] = 15.0
        return off
    return np.zeros(K)


def _raw_activations(wl: Workload, layer_index: int, K: int, rows: int,
                     role: int, idx: int) -> np.ndarray:
    """float32 [rows, K] before the fp16 cast, for the independent recipes."""
    g = rng(wl, layer_index, role, idx)
    ch = outlier_channels(wl, layer_index, K)
    off = channel_offsets(wl, layer_index, K).astype(np.float32)
    if wl.dist == "laplace_x100":
        x = g.laplace(0.0, 1.0, size=(rows, K)).astype(np.float32)
    else:
        x = g.standard_normal(size=(rows, K), dtype=np.float32)
    gain = {"normal_fixed8": 40.0, "normal_x60": 60.0, "offset_x50": 50.0,
            "laplace_x100": 100.0}[wl.dist]
    x[:, ch] *= np.float32(gain)
    x += off[None, :]
    return x


def weight(wl: Workload, layer_index: int) -> np.ndarray:
    """fp16 [N, K] in nn.Linear layout (in-features contiguous)."""
    lay = wl.layers[layer_index]
    g = rng(wl, layer_index, ROLE_WEIGHT)
    w = g.standard_normal(size=(lay.N, lay.K), dtype=np.float32)
    w *= np.float32(wl.w_std)
    return w.astype(np.float16)


def bias(wl: Workload, layer_index: int) -> np.ndarray:
    """fp16 [N]."""
    lay = wl.layers[layer_index]
    g = rng(wl, layer_index, ROLE_BIAS)
    return (g.standard_normal(size=lay.N) * wl.b_std).astype(np.float16)


def activations(wl: Workload, layer_index: int, rows: int, role: int = ROLE_EVAL_X,
                idx: int = 0) -> np.ndarray:
    """fp16 [rows, K] input of layer ``layer_index``.

    For the OPT-6.7B workload's fc2, the input is the ReLU of fc1's output
    on the matching fc1 input batch (computed in float64 on the host, then
    rounded to fp16), so it is non-negative and asymmetric per channel.
    """
    lay = wl.layers[layer_index]
    if wl.name == "opt6.7b_w8a8" and lay.name == "fc2":
        i1 = [l.name for l in wl.layers].index("fc1")
        x1 = activations(wl, i1, rows, role, idx).astype(np.float64)
        w1 = weight(wl, i1).astype(np.float64)
        b1 = bias(wl, i1).astype(np.float64)
        h = x1 @ w1.T
        h += b1[None, :]
        np.maximum(h, 0.0, out=h)
        return h.astype(np.float16)
    return _raw_activations(wl, layer_index, lay.K, rows, role, idx).astype(np.float16)


def calibration_batches(wl: Workload, layer_index: int, rows: int | None = None,
                        batches: int | None = None):
    """Yields the seeded calibration batches (fp16 [rows, K]) of one layer."""
    rows = wl.calib_rows if rows is None else rows
    batches = wl.calib_batches if batches is None else batches
    for i in range(batches):
        yield activations(wl, layer_index, rows, ROLE_CALIB_X, i)


# --------------------------------------------------------------------------
# LayerNorm inputs (for the linears that follow a LayerNorm: qkv and fc1)
# --------------------------------------------------------------------------
def ln_params(wl: Workload, layer_index: int):
    """fp16 gamma, beta [K] of the LayerNorm in front of layer ``layer_index``.

    gamma ~ U(0.5, 1.5) and beta ~ N(0, 0.2^2), except on the layer's outlier
    channels, where gamma ~ U(10, 30) and beta ~ U(-10, 10): the LayerNorm's
    gain is what turns a few channels into structured outliers of the
    linear's input, and its bias makes them asymmetric."""
    K = wl.layers[layer_index].K
    g = rng(wl, layer_index, ROLE_LN_PARAMS)
    gamma = g.uniform(0.5, 1.5, size=K)
    beta = g.normal(0.0, 0.2, size=K)
    ch = outlier_channels(wl, layer_index, K)
    gamma[ch] = g.uniform(10.0, 30.0, size=ch.size)
    beta[ch] = g.uniform(-10.0, 10.0, size=ch.size)
    return gamma.astype(np.float16), beta.astype(np.float16)


def ln_inputs(wl: Workload, layer_index: int, rows: int, idx: int = 0) -> np.ndarray:
    """fp16 [rows, K] LayerNorm input (the residual stream): per channel k,
    N(mu_k, sigma_k^2) with sigma_k ~ U(0.5, 2) and mu_k ~ N(0, 0.5^2), the
    layer's outlier channels with sigma_k = 20 and mu_k ~ U(-40, 40).  The
    channel moments are fixed per layer; ``idx`` 0 is the evaluated batch,
    1.. the calibration batches."""
    K = wl.layers[layer_index].K
    gp = rng(wl, layer_index, ROLE_LN_PARAMS, 1)
    sigma = gp.uniform(0.5, 2.0, size=K)
    mu = gp.normal(0.0, 0.5, size=K)
    ch = outlier_channels(wl, layer_index, K)
    sigma[ch] = 20.0
    mu[ch] = gp.uniform(-40.0, 40.0, size=ch.size)
    g = rng(wl, layer_index, ROLE_LN_INPUT, idx)
    x = g.standard_normal(size=(rows, K), dtype=np.float32)
    x *= sigma.astype(np.float32)[None, :]
    x += mu.astype(np.float32)[None, :]
    return x.astype(np.float16)

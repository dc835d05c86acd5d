"""CPU oracle for OutlierTune's per-channel-quantized linear layer.

TEST INFRASTRUCTURE ONLY.  This module is the parity reference that the HIP
library is checked against.  Only the test suite, the package's smoke check
and the benchmark's CPU-baseline leg may import it; the product path never
calls it and shares no code with it.

It is written for obviousness, not speed: plain numpy, float64 wherever the
method leaves the precision open, every rounding spelled out.  The paper
(OutlierTune, Wang et al., 2024) fixes the algebra; where it leaves a choice
open the reading taken here is noted at the function that makes it.

Notation follows the paper.  X is [M x K] (tokens x input channels), the
linear's weight W is stored as nn.Linear stores it, [N x K] (so the paper's
W^T is its transpose), b is [N].  ``qa`` and ``qw`` are the largest codes of
the activation and weight quantizers, 2^(bits-1) - 1 (symmetric, signed).

Functions and the passages they follow
--------------------------------------
calibrate       Sec. 3.2 (symmetrization factor z from per-channel max/min)
                and App. A (static min-max calibration of activations).
scales_from_minmax  the same scales from a stored calibration state, for
                another bit-width or without symmetrization (Sec. 4.4).
fold_weights    Sec. 3.1, Eq. (e) (W_s = W scaled by s^X along input
                channels), Eq. (f) (per-output-channel quantization of W_s),
                Sec. 3.2, Eq. (g) (shift z moved into the bias: z W^T + b),
                and the Implementation paragraph (weights quantized offline).
quantize_act    Eq. (g): round((X - z) / s^X), per input channel.
int_gemm        Eq. (f) right-hand side: the integer sum over k.
epilogue        Eq. (g): scale by s^{W_s}_j, then add (z W^T + b).
qlinear         int_gemm followed by epilogue.
internal_scaling_fp64   Eq. (d) with unrounded operands (used by the tests).
layernorm_stats Row mean and variance of the LayerNorm that precedes the
                linear (Sec. 3.2, Implementation paragraph: quantization
                fused with the preceding LayerNorm).
ln_scaled_act   LayerNorm with the shift z taken into its bias (Sec. 3.2:
                z combined with the LayerNorm bias), divided by s per
                channel, without an fp16 round trip.
ln_quantize_act Eq. (g)'s per-channel codes of that value.
quantize_act_per_token  Eq. (c): dynamic per-token scales s^X_m for the
                linears without activation outliers (out, fc2; Sec. 3.2
                and Sec. 4.1), and the codes round(X / s^X).
fold_weights_per_token  Eq. (c) and Eq. (h): per-output-channel weight
                scales without an activation scale, and the bias b + z that
                carries a symmetrized residual stream back (Eq. (h)).
epilogue_per_token      Eq. (c): s^X_m s^W_n times the integer sum, plus b'.
fold_weights_asym       the "Int8" weight setting (Sec. 4.1, App. A):
                per-output-channel asymmetric quantization of W_s with a zero
                point, Eq. (a) with z != 0.
int_gemm_asym   Eq. (f)'s integer sum with the weight zero point removed:
                sum_k Xq (Wq - zW).
reference_fp64, folded_fp64     exact-arithmetic references (tests only).

Readings taken where the paper is silent (each applies to both this oracle
and the HIP path):
  * The rounding operation of Eq. (a) is round-half-to-even.
  * Quantization is symmetric and signed: codes lie in [-q, q] with
    q = 2^(bits-1) - 1 (Eq. (a) with zero point 0, range made signed).
  * Divisions by a scale are carried out as a float32 multiply by a stored
    reciprocal for activations, and as a correctly rounded float64 division
    for weights.
  * Scales and shifts are computed in float64 and stored in float32.
  * The activation scale is half the calibrated range over qa, so the
    calibration extremes map to exactly -qa and +qa after symmetrization.
  * A constant channel (range 0) gets scale 1; an all-zero weight row gets
    weight scale 1.
  * The compensated bias is kept in float32.
  * Minimum and maximum treat -0 as +0.
  * LayerNorm statistics (population variance, divisor K) come from exact
    integer sums of the fp16 inputs scaled by 2^24; mean and variance are
    then rounded to float64 in the order spelled out in layernorm_stats, and
    the per-element normalization runs in float32 (see ln_quantize_act).
"""
from __future__ import annotations

import math

import numpy as np

INT32_LIMIT = 2 ** 31


class NonFinite(ValueError):
    """Raised when calibration data or weights contain NaN or infinity."""


def qmax(bits: int) -> int:
    """Largest code of a signed symmetric ``bits``-bit quantizer (Eq. (a))."""
    if not 2 <= int(bits) <= 8:
        raise ValueError(f"bits must be in [2, 8], got {bits}")
    return (1 << (int(bits) - 1)) - 1


# --------------------------------------------------------------------------
# O1: calibration (Sec. 3.2; App. A)
# --------------------------------------------------------------------------
def calibrate(batches, a_bits: int):
    """Static per-channel min-max calibration and symmetrization factors.

    For every input channel k, over all rows of all calibration batches:
      lo_k, hi_k  = min and max of the channel (fp16 values, exact in fp64);
      z_k         = (hi_k + lo_k) / 2            -- Sec. 3.2's shift;
      s_k         = ((hi_k - lo_k) / 2) / qa     -- min-max scale of X - z;
      inv_s_k     = 1 / s_k.
    z, s and inv_s are computed in float64 and stored as float32; a channel
    with hi_k == lo_k (or a scale that underflows float32) gets s_k = 1.

    Returns (minmax, z, s, inv_s): minmax is float32 [2K], the K minima
    followed by the K maxima (fp16 values, so exact in float32).
    """
    qa = qmax(a_bits)
    lo = hi = None
    for x in batches:
        x = np.asarray(x)
        if x.dtype != np.float16 or x.ndim != 2 or x.shape[0] == 0:
            raise ValueError("calibration batches must be non-empty fp16 [rows, K]")
        x64 = x.astype(np.float64) + 0.0  # "+ 0.0" turns -0 into +0
        if not np.all(np.isfinite(x64)):
            raise NonFinite("non-finite calibration data")
        bmin = x64.min(axis=0)
        bmax = x64.max(axis=0)
        lo = bmin if lo is None else np.minimum(lo, bmin)
        hi = bmax if hi is None else np.maximum(hi, bmax)
    if lo is None:
        raise ValueError("no calibration batches")
    z = ((hi + lo) / 2.0).astype(np.float32)
    half = (hi - lo) / 2.0
    s = (half / float(qa)).astype(np.float32)
    s[s == 0] = np.float32(1.0)
    inv_s = (1.0 / s.astype(np.float64)).astype(np.float32)
    minmax = np.concatenate([lo, hi]).astype(np.float32)
    return minmax, z, s, inv_s


def scales_from_minmax(minmax, a_bits: int, symmetrize: bool = True):
    """(z, s, inv_s) from a calibration state minmax [2K] (the K minima then
    the K maxima, as calibrate returns it), for ``a_bits`` codes.

    With symmetrization (Sec. 3.2) this is calibrate's rule: z = (hi + lo)/2,
    s = ((hi - lo)/2)/qa.  Without it (the ablation of Sec. 4.4, Table 6)
    the range is not shifted: z = 0 and s = max(|lo|, |hi|)/qa, so the
    larger side of the range lands on +-qa and the other side wastes codes.
    float64 math, float32 storage; s = 1 where it would be 0.
    """
    qa = qmax(a_bits)
    mm = np.asarray(minmax, dtype=np.float32).astype(np.float64)
    K = mm.size // 2
    lo, hi = mm[:K], mm[K:]
    if symmetrize:
        z = ((hi + lo) / 2.0).astype(np.float32)
        s = (((hi - lo) / 2.0) / float(qa)).astype(np.float32)
    else:
        z = np.zeros(K, dtype=np.float32)
        s = (np.maximum(np.abs(lo), np.abs(hi)) / float(qa)).astype(np.float32)
    s[s == 0] = np.float32(1.0)
    inv_s = (1.0 / s.astype(np.float64)).astype(np.float32)
    return z, s, inv_s


# --------------------------------------------------------------------------
# O2: offline weight transform (Eq. (e), (f), (g); Implementation paragraph)
# --------------------------------------------------------------------------
def fold_weights(W, b, z, s, w_bits: int):
    """Fold the activation scale into W, quantize per output channel, and
    move the symmetrization shift into the bias.

      W_s[n, k]  = W[n, k] * s_k                      Eq. (e) (exact in fp64)
      sW_n       = max_k |W_s[n, k]| / qw              min-max, per out channel
      Wq[n, k]   = clip(round(W_s[n, k] / sW_n), -qw, qw)           Eq. (f)
      b'_n       = sum_k z_k * W[n, k] + b_n   (original W)         Eq. (g)

    The sum for b'_n runs over k in ascending order in float64 (each product
    is exact), b_n is added last, and the result is stored as float32.
    ``b`` may be None (no bias).  Returns (Wq int8 [N, K], sW float32 [N],
    bprime float32 [N]).
    """
    qw = qmax(w_bits)
    W = np.asarray(W)
    if W.dtype != np.float16 or W.ndim != 2:
        raise ValueError("W must be fp16 [N, K]")
    N, K = W.shape
    W64 = W.astype(np.float64)
    b64 = np.zeros(N) if b is None else np.asarray(b).astype(np.float64)
    if not (np.all(np.isfinite(W64)) and np.all(np.isfinite(b64))):
        raise NonFinite("non-finite weights or bias")
    s64 = np.asarray(s, dtype=np.float32).astype(np.float64)
    z64 = np.asarray(z, dtype=np.float32).astype(np.float64)
    assert s64.shape == (K,) and z64.shape == (K,)

    Ws = W64 * s64[None, :]
    m = np.abs(Ws).max(axis=1)
    sW = (m / float(qw)).astype(np.float32)
    sW[sW == 0] = np.float32(1.0)
    Wq = np.clip(np.rint(Ws / sW.astype(np.float64)[:, None]), -qw, qw).astype(np.int8)

    acc = np.zeros(N)
    for k in range(K):
        acc = acc + z64[k] * W64[:, k]
    bprime = (acc + b64).astype(np.float32)
    return Wq, sW, bprime


# --------------------------------------------------------------------------
# O3: runtime activation quantization (Eq. (g))
# --------------------------------------------------------------------------
def quantize_act(X, z, inv_s, a_bits: int):
    """Codes of the symmetrized activations, per input channel:

      t = fp32(X) - z_k        (float32, round to nearest even)
      u = t * inv_s_k          (float32, round to nearest even)
      q = clip(round(u), -qa, qa)

    Values outside the calibrated range clip to +-qa.
    """
    qa = qmax(a_bits)
    X = np.asarray(X)
    if X.dtype != np.float16 or X.ndim != 2:
        raise ValueError("X must be fp16 [M, K]")
    z = np.asarray(z, dtype=np.float32)
    inv_s = np.asarray(inv_s, dtype=np.float32)
    t = X.astype(np.float32) - z[None, :]
    u = t * inv_s[None, :]
    assert u.dtype == np.float32
    return np.clip(np.rint(u), -qa, qa).astype(np.int8)


# --------------------------------------------------------------------------
# O4: integer GEMM (Eq. (f), right-hand side)
# --------------------------------------------------------------------------
def check_acc_range(K: int, a_bits: int, w_bits: int) -> None:
    """The int32 accumulator cannot overflow iff K * qa * qw < 2^31."""
    if K * qmax(a_bits) * qmax(w_bits) >= INT32_LIMIT:
        raise OverflowError("K * qa * qw must be below 2^31")


def int_gemm(Xq, Wq):
    """acc[m, n] = sum_k Xq[m, k] * Wq[n, k], exact, as int32.

    Computed as a float64 matrix product of the integer codes: every partial
    sum is an integer of magnitude at most K * 127 * 127 < 2^53, so the
    product is exact whatever order the BLAS sums in.
    """
    Xq = np.asarray(Xq)
    Wq = np.asarray(Wq)
    assert Xq.ndim == 2 and Wq.ndim == 2 and Xq.shape[1] == Wq.shape[1]
    K = Xq.shape[1]
    if K * 127 * 127 >= 2 ** 53:
        raise OverflowError("K too large for an exact float64 product")
    acc = Xq.astype(np.float64) @ Wq.astype(np.float64).T
    return acc.astype(np.int64).astype(np.int32)


# --------------------------------------------------------------------------
# O5: dequantization epilogue (Eq. (g))
# --------------------------------------------------------------------------
def epilogue_fp32(acc, sW, bprime):
    """y = fp32(fp32(fp32(acc) * sW_n) + b'_n), every step float32 RNE."""
    acc = np.asarray(acc, dtype=np.int32)
    v = acc.astype(np.float32)
    p = v * np.asarray(sW, dtype=np.float32)[None, :]
    y = p + np.asarray(bprime, dtype=np.float32)[None, :]
    assert y.dtype == np.float32
    return y


def epilogue(acc, sW, bprime):
    """Y = fp16(y) of :func:`epilogue_fp32` (round to nearest even, +-inf on
    overflow)."""
    return epilogue_fp32(acc, sW, bprime).astype(np.float16)


def qlinear(Xq, Wq, sW, bprime):
    """The quantized linear: :func:`int_gemm` then :func:`epilogue`."""
    return epilogue(int_gemm(Xq, Wq), sW, bprime)


# --------------------------------------------------------------------------
# O6: exact-arithmetic references (tests only)
# --------------------------------------------------------------------------
def reference_fp64(X, W, b):
    """The unquantized linear X W^T + b in float64."""
    X64 = np.asarray(X).astype(np.float64)
    W64 = np.asarray(W).astype(np.float64)
    out = X64 @ W64.T
    if b is not None:
        out = out + np.asarray(b).astype(np.float64)[None, :]
    return out


def folded_fp64(X, W, b, z, s):
    """Eq. (g) with every rounding removed:
    ((X - z) / s) (W * s)^T + (z W^T + b), in float64."""
    X64 = np.asarray(X).astype(np.float64)
    W64 = np.asarray(W).astype(np.float64)
    z64 = np.asarray(z).astype(np.float64)
    s64 = np.asarray(s).astype(np.float64)
    b64 = 0.0 if b is None else np.asarray(b).astype(np.float64)
    xs = (X64 - z64[None, :]) / s64[None, :]
    Ws = W64 * s64[None, :]
    return xs @ Ws.T + (z64[None, :] @ W64.T + b64)


def internal_scaling_fp64(Xt, Wt, sX, sWvec):
    """Eq. (d): Y_ij = s^W_j * sum_k s^X_k * Xt_ik * Wt_kj (Wt given as
    [N, K], i.e. the paper's W^T), float64, with the scale inside the sum."""
    Xt = np.asarray(Xt, dtype=np.float64)
    Wt = np.asarray(Wt, dtype=np.float64)
    sX = np.asarray(sX, dtype=np.float64)
    sWvec = np.asarray(sWvec, dtype=np.float64)
    M, K = Xt.shape
    N = Wt.shape[0]
    Y = np.zeros((M, N))
    for k in range(K):
        Y += sX[k] * np.outer(Xt[:, k], Wt[:, k])
    return Y * sWvec[None, :]


# --------------------------------------------------------------------------
# LayerNorm fused with symmetrization and quantization (Sec. 3.2,
# Implementation paragraph)
# --------------------------------------------------------------------------
def layernorm_stats(H):
    """Mean and population variance (divisor K) of every row of fp16 H [M, K].

    Every fp16 value is an integer multiple of 2^-24, so a_k = h_k * 2^24 is
    an exact integer (|a_k| < 2^40) and the sums S1 = sum a_k and
    S2 = sum a_k^2 are taken exactly (Python integers).  Then
      mean = fl(fl(S1) / K) * 2^-24
      var  = fl(fl(K * S2 - S1^2) / K^2) * 2^-48
    where fl() rounds to the nearest float64 (ties to even); K * S2 - S1^2
    is K^2 times the exact population variance of the a_k.  Returns two
    float64 arrays [M].
    """
    H = np.asarray(H)
    if H.dtype != np.float16 or H.ndim != 2:
        raise ValueError("H must be fp16 [M, K]")
    M, K = H.shape
    a = H.astype(np.float64) * 2.0 ** 24
    assert np.all(a == np.trunc(a))
    a = a.astype(np.int64)
    mean = np.empty(M)
    var = np.empty(M)
    for m in range(M):
        row = [int(v) for v in a[m]]
        S1 = sum(row)
        S2 = sum(v * v for v in row)
        mean[m] = float(S1) / K * 2.0 ** -24
        var[m] = float(K * S2 - S1 * S1) / float(K * K) * 2.0 ** -48
    return mean, var


def ln_scaled_act(H, gamma, beta, eps, z, inv_s):
    """The symmetrized, scaled LayerNorm output u (float32 [M, K]) that
    ln_quantize_act rounds to codes.

    The LayerNorm y = (h - mean) / sqrt(var + eps) * gamma + beta is followed
    by Eq. (g)'s quantization of y - z; with z taken into the LayerNorm's
    bias (Sec. 3.2) the symmetrized value is produced directly and never
    stored.  Per row (mean, var from layernorm_stats, eps a float32 value):
      rstd = 1 / sqrt(var + eps)        float64, each step rounded to nearest
      mu32, r32 = fp32(mean), fp32(rstd)
    and per element, every step a float32 operation rounded to nearest even:
      d = fp32(h) - mu32;  n = d * r32;  g = n * fp32(gamma_k)
      c = fp32(beta_k) - z_k            (the shifted LayerNorm bias)
      y = g + c;  u = y * inv_s_k
    """
    H = np.asarray(H)
    mean, var = layernorm_stats(H)
    M, K = H.shape
    gamma = np.asarray(gamma)
    beta = np.asarray(beta)
    if gamma.dtype != np.float16 or beta.dtype != np.float16 or gamma.shape != (K,) \
            or beta.shape != (K,):
        raise ValueError("gamma and beta must be fp16 [K]")
    eps64 = float(np.float32(eps))
    rstd = np.array([1.0 / math.sqrt(v + eps64) for v in var])
    mu32 = mean.astype(np.float32)[:, None]
    r32 = rstd.astype(np.float32)[:, None]
    z = np.asarray(z, dtype=np.float32)
    inv_s = np.asarray(inv_s, dtype=np.float32)
    c = beta.astype(np.float32) - z
    d = H.astype(np.float32) - mu32
    n = d * r32
    g = n * gamma.astype(np.float32)[None, :]
    y = g + c[None, :]
    u = y * inv_s[None, :]
    assert u.dtype == np.float32
    return u


def ln_quantize_act(H, gamma, beta, eps, z, inv_s, a_bits: int):
    """Codes of the symmetrized LayerNorm output, per input channel:
    q = clip(round(u), -qa, qa) with u from ln_scaled_act.  int8 [M, K]."""
    qa = qmax(a_bits)
    u = ln_scaled_act(H, gamma, beta, eps, z, inv_s)
    return np.clip(np.rint(u), -qa, qa).astype(np.int8)


# --------------------------------------------------------------------------
# Per-token path for the linears without activation outliers (Eq. (c), (h))
# --------------------------------------------------------------------------
def quantize_act_per_token(X, a_bits: int):
    """Dynamic per-token symmetric quantization, Eq. (c) (Sec. 4.1: per-token
    symmetric for the activations that are not LayerNorm outputs).

    Per row m: s_m = fp32(max_k |x_mk| / qa) (float64 division; s_m = 1 for
    a row of zeros), inv_m = fp32(1 / s_m) (float64), and
      q = clip(round(fp32(x) * inv_m), -qa, qa)   (float32 multiply, RNE).
    Returns (Xq int8 [M, K], s float32 [M]).
    """
    qa = qmax(a_bits)
    X = np.asarray(X)
    if X.dtype != np.float16 or X.ndim != 2:
        raise ValueError("X must be fp16 [M, K]")
    mx = np.abs(X.astype(np.float64)).max(axis=1)
    s = (mx / float(qa)).astype(np.float32)
    s[s == 0] = np.float32(1.0)
    inv = (1.0 / s.astype(np.float64)).astype(np.float32)
    u = X.astype(np.float32) * inv[:, None]
    assert u.dtype == np.float32
    return np.clip(np.rint(u), -qa, qa).astype(np.int8), s


def fold_weights_per_token(W, b, zres, w_bits: int):
    """Weights of a per-token linear (Eq. (c)): no activation scale to fold.

      sW_n = max_k |W[n, k]| / qw        (float64, stored float32; 1 for a
                                          zero row)
      Wq   = clip(round(W / sW_n), -qw, qw)     correctly rounded fp64 division
      b'_n = b_n + zres_n                 Eq. (h): with a symmetrized residual
                                          stream X_res - z, its shift z comes
                                          back through the bias
    ``b`` and ``zres`` may be None (zero).  b' is summed in float64 and
    stored float32.  Returns (Wq int8 [N, K], sW float32 [N], b' float32 [N]).
    """
    qw = qmax(w_bits)
    W = np.asarray(W)
    if W.dtype != np.float16 or W.ndim != 2:
        raise ValueError("W must be fp16 [N, K]")
    N, K = W.shape
    W64 = W.astype(np.float64)
    b64 = np.zeros(N) if b is None else np.asarray(b).astype(np.float64)
    if not (np.all(np.isfinite(W64)) and np.all(np.isfinite(b64))):
        raise NonFinite("non-finite weights or bias")
    z64 = np.zeros(N) if zres is None else np.asarray(zres, dtype=np.float32).astype(np.float64)
    assert z64.shape == (N,)
    sW = (np.abs(W64).max(axis=1) / float(qw)).astype(np.float32)
    sW[sW == 0] = np.float32(1.0)
    Wq = np.clip(np.rint(W64 / sW.astype(np.float64)[:, None]), -qw, qw).astype(np.int8)
    bprime = (b64 + z64).astype(np.float32)
    return Wq, sW, bprime


def epilogue_per_token(acc, sX, sW, bprime):
    """Eq. (c) with the bias: y = fp16(fp32(fp32(fp32(acc) * sX_m) * sW_n)
    + b'_n), each float32 operation rounded to nearest even."""
    a = np.asarray(acc, dtype=np.int64).astype(np.float32)
    t = a * np.asarray(sX, dtype=np.float32)[:, None]
    p = t * np.asarray(sW, dtype=np.float32)[None, :]
    y = p + np.asarray(bprime, dtype=np.float32)[None, :]
    assert y.dtype == np.float32
    return y.astype(np.float16)


# --------------------------------------------------------------------------
# Asymmetric per-channel weights, the paper's "Int8" setting (Sec. 4.1,
# App. A), with Eq. (a)'s zero point
# --------------------------------------------------------------------------
def fold_weights_asym(W, b, z, s, w_bits: int):
    """Fold s into W (Eq. (e)) and quantize each output channel of W_s
    asymmetrically, Eq. (a): codes c = clip(round(W_s / sW) + zW, 0, L),
    L = 2^bits - 1, dequantized as (c - zW) sW.

      lo_n, hi_n = min(min_k W_s[n, k], 0), max(max_k W_s[n, k], 0)
                   (the range always holds 0, so 0 is represented exactly)
      sW_n = fp32((hi_n - lo_n) / L)        (float64; 1 where it is 0)
      zW_n = clip(round(-lo_n / sW_n), 0, L)
    Codes are stored signed, shifted by 2^(bits-1) so that they fit int8 for
    the int8 matrix cores: Wq = c - 2^(bits-1), zWq = zW - 2^(bits-1).  The
    bias b' = z W^T + b is the symmetric path's (original W, Eq. (g)).
    Returns (Wq int8 [N, K], sW float32 [N], zWq int32 [N], b' float32 [N]).
    """
    L = (1 << int(w_bits)) - 1
    half = 1 << (int(w_bits) - 1)
    qmax(w_bits)  # validates the bit-width
    W = np.asarray(W)
    if W.dtype != np.float16 or W.ndim != 2:
        raise ValueError("W must be fp16 [N, K]")
    N, K = W.shape
    W64 = W.astype(np.float64)
    b64 = np.zeros(N) if b is None else np.asarray(b).astype(np.float64)
    if not (np.all(np.isfinite(W64)) and np.all(np.isfinite(b64))):
        raise NonFinite("non-finite weights or bias")
    s64 = np.asarray(s, dtype=np.float32).astype(np.float64)
    z64 = np.asarray(z, dtype=np.float32).astype(np.float64)
    Ws = W64 * s64[None, :]
    lo = np.minimum(Ws.min(axis=1), 0.0)
    hi = np.maximum(Ws.max(axis=1), 0.0)
    sW = ((hi - lo) / float(L)).astype(np.float32)
    sW[sW == 0] = np.float32(1.0)
    sW64 = sW.astype(np.float64)
    zW = np.clip(np.rint(-lo / sW64), 0, L)
    c = np.clip(np.rint(Ws / sW64[:, None]) + zW[:, None], 0, L)
    Wq = (c - half).astype(np.int8)
    zWq = (zW - half).astype(np.int32)
    acc = np.zeros(N)
    for k in range(K):
        acc = acc + z64[k] * W64[:, k]
    bprime = (acc + b64).astype(np.float32)
    return Wq, sW, zWq, bprime


def int_gemm_asym(Xq, Wq, zWq):
    """acc[m, n] = sum_k Xq[m, k] (Wq[n, k] - zWq[n]), exact (float64 BLAS on
    integers below 2^53), as int32.  The shift of the stored codes cancels:
    Wq - zWq = c - zW."""
    Xq = np.asarray(Xq)
    Wd = np.asarray(Wq).astype(np.int64) - np.asarray(zWq, dtype=np.int64)[:, None]
    acc = Xq.astype(np.float64) @ Wd.astype(np.float64).T
    assert np.all(np.abs(acc) < INT32_LIMIT)
    return acc.astype(np.int32)


def pipeline(X, W, b, calib_batches, a_bits: int, w_bits: int):
    """Calibrate, fold, quantize and run the quantized linear end to end.
    Returns a dict of every intermediate."""
    minmax, z, s, inv_s = calibrate(calib_batches, a_bits)
    Wq, sW, bprime = fold_weights(W, b, z, s, w_bits)
    Xq = quantize_act(X, z, inv_s, a_bits)
    check_acc_range(Xq.shape[1], a_bits, w_bits)
    acc = int_gemm(Xq, Wq)
    Y = epilogue(acc, sW, bprime)
    return dict(minmax=minmax, z=z, s=s, inv_s=inv_s, Wq=Wq, sW=sW,
                bprime=bprime, Xq=Xq, acc=acc, Y=Y)

"""GPU parity of ot_ln_quantize_act (LayerNorm fused with symmetrization and
per-channel quantization, Sec. 3.2) against the CPU oracle, through the C
ABI: codes bit for bit.

The kernel takes the row statistics on a float64 fast path with a proven
error bound and falls back to exact integer sums for the rows the bound
cannot settle; the oracle takes them exactly.  Besides random and workload
rows, the cases below build rows that must take the fallback (a mean of
exactly 0, a mean exactly halfway between two fp32 values) and give each
row a channel where a one-unit change of fp32(mean) or fp32(rstd) moves the
code by about 20, so a wrong rounding cannot hide."""
import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import ot, synth

pytestmark = pytest.mark.gpu


def case(msg):
    print(f"[case] {msg}", flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _textbook_ln_fp16(H, gamma, beta, eps):
    """fp16 LayerNorm output (numpy float64), the data calibration sees."""
    h = H.astype(np.float64)
    y = (h - h.mean(1, keepdims=True)) / np.sqrt(h.var(1, keepdims=True) + eps)
    return (y * gamma.astype(np.float64) + beta.astype(np.float64)).astype(np.float16)


def _random_inputs(M, K, seed, a_bits=8, eps=1e-5):
    r = np.random.default_rng(seed)
    sigma = r.uniform(0.3, 3.0, K)
    mu = r.normal(0, 2.0, K)
    out = r.choice(K, size=max(1, K // 100), replace=False)
    sigma[out] *= 20
    H = (r.standard_normal((M, K)) * sigma + mu).astype(np.float16)
    gamma = r.uniform(0.5, 1.5, K)
    gamma[out] = r.uniform(5, 20, out.size)
    gamma = gamma.astype(np.float16)
    beta = r.normal(0, 0.5, K).astype(np.float16)
    calib = (r.standard_normal((64, K)) * sigma + mu).astype(np.float16)
    _, z, s, inv_s = O.calibrate([_textbook_ln_fp16(calib, gamma, beta, eps)], a_bits)
    return H, gamma, beta, z, inv_s


def assert_codes_match(got, H, gamma, beta, eps, z, inv_s, a_bits):
    ref = O.ln_quantize_act(H, gamma, beta, eps, z, inv_s, a_bits)
    assert got.shape == ref.shape
    differ = got != ref
    assert not differ.any(), (f"{int(differ.sum())} of {differ.size} codes differ, rows "
                              f"{np.unique(np.nonzero(differ)[0])[:10]}")


def _run(H, gamma, beta, eps, a_bits, z, inv_s):
    Xq = ot.ln_quantize_act(dev(H), dev(gamma), dev(beta), eps, a_bits, dev(z), dev(inv_s))
    torch.cuda.synchronize()
    return Xq.cpu().numpy()


# widths on both sides of the 49152 kernel-configuration boundary (6 and 8
# chunks of 8 channels per thread), ragged against the 8-channel chunks and
# the 64-thread waves, up to the widest row
SHAPES = [(1, 16), (3, 768), (17, 1040), (130, 512), (4, 2048), (7, 2064), (64, 4096),
          (9, 5120), (5, 16384),
          (2, 16400), (3, 32768), (2, 32784), (2, 49152), (2, 49168), (1, 65536)]


@pytest.mark.parametrize("M,K", SHAPES)
def test_parity_random(M, K):
    case(f"ln_quantize M={M} K={K}")
    H, gamma, beta, z, inv_s = _random_inputs(M, K, 100 * M + K)
    got = _run(H, gamma, beta, 1e-5, 8, z, inv_s)
    assert_codes_match(got, H, gamma, beta, 1e-5, z, inv_s, 8)


@pytest.mark.parametrize("a_bits", [6, 4, 2])
def test_parity_low_bits(a_bits):
    case(f"ln_quantize a_bits={a_bits}")
    H, gamma, beta, z, inv_s = _random_inputs(40, 2064, 7 + a_bits, a_bits)
    got = _run(H, gamma, beta, 1e-5, a_bits, z, inv_s)
    assert_codes_match(got, H, gamma, beta, 1e-5, z, inv_s, a_bits)
    assert np.abs(got).max() <= O.qmax(a_bits)


def test_parity_extreme_rows():
    """Largest fp16 magnitudes (128-bit sums with a high word), subnormals,
    zero and constant rows, a single spike, alternating extremes."""
    case("ln_quantize extreme rows")
    K = 1024
    r = np.random.default_rng(3)
    rows = [
        np.full(K, 65504.0), np.full(K, -65504.0),
        np.where(np.arange(K) % 2 == 0, 65504.0, -65504.0),
        np.zeros(K), np.full(K, 3.0),
        r.integers(-1023, 1024, K) * 2.0 ** -24,  # subnormals only
        np.concatenate([[60000.0], np.full(K - 1, 2.0 ** -24)]),
        np.clip(r.standard_normal(K) * 20000.0, -65504.0, 65504.0),
        np.where(r.random(K) < 0.5, 6.0e-8, 65000.0),
    ]
    H = np.stack(rows).astype(np.float16)
    assert np.all(np.isfinite(H.astype(np.float32)))
    gamma = r.uniform(0.5, 1.5, K).astype(np.float16)
    beta = r.normal(0, 1, K).astype(np.float16)
    z = r.normal(0, 0.5, K).astype(np.float32)
    inv_s = r.uniform(10, 40, K).astype(np.float32)
    for eps in (1e-5, 1e-12, 1.0):
        got = _run(H, gamma, beta, eps, 8, z, inv_s)
        assert_codes_match(got, H, gamma, beta, eps, z, inv_s, 8)


def test_eps_zero_on_rows_with_spread():
    case("ln_quantize eps=0")
    H, gamma, beta, z, inv_s = _random_inputs(16, 768, 21)
    assert_codes_match(_run(H, gamma, beta, 0.0, 8, z, inv_s), H, gamma, beta, 0.0, z, inv_s, 8)


@pytest.mark.parametrize("name,li", [("opt125m_w8a8", 0), ("opt6.7b_w8a8", 2),
                                     ("opt13b_w6a6", 0), ("opt66b_w8a8", 0)])
def test_parity_workload_inputs(name, li):
    """The seeded LayerNorm inputs of the workloads, calibrated on the fp16
    LayerNorm output of their calibration rows."""
    wl = synth.WORKLOADS[name]
    K = wl.layers[li].K
    case(f"ln_quantize {name}/{wl.layers[li].name} K={K}")
    gamma, beta = synth.ln_params(wl, li)
    calib = [_textbook_ln_fp16(synth.ln_inputs(wl, li, 128, 1 + i), gamma, beta, 1e-5)
             for i in range(2)]
    _, z, s, inv_s = O.calibrate(calib, wl.a_bits)
    H = synth.ln_inputs(wl, li, 24)
    got = _run(H, gamma, beta, 1e-5, wl.a_bits, z, inv_s)
    assert_codes_match(got, H, gamma, beta, 1e-5, z, inv_s, wl.a_bits)


def test_fullsize_opt13b_qkv_input_every_row():
    """4096 x 5120 (the OPT-13B qkv input): every code against the oracle,
    and the run repeated gives identical bytes."""
    wl = synth.WORKLOADS["opt13b_w6a6"]
    K, M = wl.layers[0].K, wl.M
    case(f"ln_quantize fullsize M={M} K={K}")
    gamma, beta = synth.ln_params(wl, 0)
    calib = [_textbook_ln_fp16(synth.ln_inputs(wl, 0, 256, 1), gamma, beta, 1e-5)]
    _, z, s, inv_s = O.calibrate(calib, wl.a_bits)
    H = synth.ln_inputs(wl, 0, M)
    args = (dev(H), dev(gamma), dev(beta), 1e-5, wl.a_bits, dev(z), dev(inv_s))
    Xq = ot.ln_quantize_act(*args)
    Xq2 = ot.ln_quantize_act(*args)
    torch.cuda.synchronize()
    assert torch.equal(Xq, Xq2)
    got = Xq.cpu().numpy()
    assert int(np.abs(got).max()) <= O.qmax(wl.a_bits)
    assert_codes_match(got, H, gamma, beta, 1e-5, z, inv_s, wl.a_bits)


def _sensitive(H, gamma, beta, z, inv_s, eps):
    """Gives row m its own channel j = 1 + m where the code moves by about 20
    if fp32(mean) or fp32(rstd) of that row is off by one unit: a gain of
    65504, a reciprocal scale of 1e4, and a shift that brings the row's
    value there near 0.  Uses the oracle's statistics (test input only)."""
    gamma, beta, z, inv_s = gamma.copy(), beta.copy(), z.copy(), inv_s.copy()
    mean, var = O.layernorm_stats(H)
    mu32 = mean.astype(np.float32)
    r32 = (1.0 / np.sqrt(var + float(np.float32(eps)))).astype(np.float32)
    for m in range(H.shape[0]):
        j = 1 + m
        gamma[j] = np.float16(65504.0)
        beta[j] = np.float16(0.0)
        inv_s[j] = np.float32(1e4)
        g = ((H[m, j].astype(np.float32) - mu32[m]) * r32[m]) * np.float32(65504.0)
        z[j] = np.float32(g) + np.float32(3e-4)
    return gamma, beta, z, inv_s


def _zero_mean_rows(r, M, K):
    """Rows whose values cancel in pairs: the mean is exactly 0, the spread
    is not, so the float64 bound can never settle fp32(mean)."""
    rows = []
    for i in range(M):
        half = (r.standard_normal(K // 2) * r.uniform(0.05, 30.0)).astype(np.float16)
        row = np.concatenate([half, -half])
        r.shuffle(row)
        rows.append(row)
    return np.stack(rows).astype(np.float16)


def _tie_mean_rows(r, M, K, first_channel):
    """Rows whose exact mean lies halfway between two adjacent fp32 values,
    tuned with one subnormal element (a step of 2^-24 in the row sum).  Row
    i holds a value near its mean at channel first_channel + i, where a
    one-unit change of fp32(mean) then changes h - mean exactly."""
    from fractions import Fraction
    rows = []
    while len(rows) < M:
        off = r.uniform(0.26, 0.49)
        row = (r.standard_normal(K) + off).astype(np.float16)
        row[first_channel + len(rows)] = np.float16(off)
        row[-1] = 0
        a = row.astype(np.float64) * 2.0 ** 24
        S = int(a.astype(np.int64).sum())
        m0 = Fraction(S, K * 2 ** 24)
        f = np.float32(float(m0))
        up = np.nextafter(f, np.float32(np.inf))
        dn = np.nextafter(f, np.float32(-np.inf))
        mid = min((Fraction(float(f)) + Fraction(float(up))) / 2,
                  (Fraction(float(f)) + Fraction(float(dn))) / 2, key=lambda v: abs(v - m0))
        need = mid * K * 2 ** 24 - S
        if need.denominator != 1 or abs(need) > 1023:
            continue
        row[-1] = np.float16(int(need) * 2.0 ** -24)
        assert Fraction(int((row.astype(np.float64) * 2.0 ** 24).astype(np.int64).sum()),
                        K * 2 ** 24) == mid
        rows.append(row)
    return np.stack(rows).astype(np.float16)


@pytest.mark.parametrize("K", [1024, 5120])
def test_exact_fallback_rows(K):
    """Rows the float64 bound cannot settle, mixed with ordinary rows, each
    with a channel that exposes a one-unit error of fp32(mean) or
    fp32(rstd)."""
    case(f"ln_quantize exact-fallback rows K={K}")
    r = np.random.default_rng(K)
    H = np.concatenate([_zero_mean_rows(r, 12, K), _tie_mean_rows(r, 12, K, 13),
                        (r.standard_normal((12, K)) * 3 + 0.4).astype(np.float16)])
    gamma = r.uniform(0.5, 1.5, K).astype(np.float16)
    beta = r.normal(0, 0.5, K).astype(np.float16)
    z = r.normal(0, 0.3, K).astype(np.float32)
    inv_s = r.uniform(10, 40, K).astype(np.float32)
    for eps in (1e-5, 0.0):
        g2, b2, z2, i2 = _sensitive(H, gamma, beta, z, inv_s, eps)
        got = _run(H, g2, b2, eps, 8, z2, i2)
        assert_codes_match(got, H, g2, b2, eps, z2, i2, 8)
        # the sensitive channels are in range, so they do test the rounding
        u = O.ln_scaled_act(H, g2, b2, eps, z2, i2)
        idx = np.arange(H.shape[0])
        assert np.all(np.abs(u[idx, 1 + idx]) < 100)


@pytest.mark.parametrize("name,li", [("opt13b_w6a6", 2), ("opt66b_w8a8", 0)])
def test_workload_rows_sensitive(name, li):
    """Workload LayerNorm inputs (the fast path nearly always) with the
    sensitive channels."""
    wl = synth.WORKLOADS[name]
    K = wl.layers[li].K
    case(f"ln_quantize sensitive {name}/{wl.layers[li].name} K={K}")
    gamma, beta = synth.ln_params(wl, li)
    calib = [_textbook_ln_fp16(synth.ln_inputs(wl, li, 128, 1), gamma, beta, 1e-5)]
    _, z, s, inv_s = O.calibrate(calib, 8)
    H = synth.ln_inputs(wl, li, 64)
    g2, b2, z2, i2 = _sensitive(H, gamma, beta, z, inv_s, 1e-5)
    got = _run(H, g2, b2, 1e-5, 8, z2, i2)
    assert_codes_match(got, H, g2, b2, 1e-5, z2, i2, 8)


def test_close_to_unfused_layernorm_then_quantize():
    """Fused codes against torch's fp32 LayerNorm rounded to fp16 followed by
    ot_quantize_act: the fused path skips that fp16 rounding, so codes may
    differ by one where the fp16 rounding crosses a rounding boundary."""
    case("ln_quantize vs unfused")
    H, gamma, beta, z, inv_s = _random_inputs(256, 2048, 5)
    got = _run(H, gamma, beta, 1e-5, 8, z, inv_s)
    h = dev(H)
    X = torch.nn.functional.layer_norm(h.float(), (2048,), dev(gamma).float(), dev(beta).float(),
                                       1e-5).half()
    unfused = ot.quantize_act(X, 8, dev(z), dev(inv_s)).cpu().numpy()
    d = np.abs(got.astype(int) - unfused)
    assert d.max() <= 1 and (d > 0).mean() < 0.1


def test_rejects_too_wide_rows():
    h = torch.zeros((2, 65536 + 16), dtype=torch.float16, device="cuda")
    p = torch.zeros(65536 + 16, dtype=torch.float16, device="cuda")
    f = torch.zeros(65536 + 16, dtype=torch.float32, device="cuda")
    with pytest.raises(ot.OTError):
        ot.ln_quantize_act(h, p, p, 1e-5, 8, f, f)

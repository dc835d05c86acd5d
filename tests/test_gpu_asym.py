"""GPU parity of the asymmetric ("Int8") weight path (ot_fold_weights_asym,
ot_qlinear_asym) against the CPU oracle, through the C ABI: codes, scales
and zero points bit-exact, b' within 1 fp32 ulp, the integer sums (with the
zero point removed) bit-exact, Y within 2 fp16 ulp and 1e-3 relative."""
import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import ot, synth
from tests._tol import assert_fp16_close, assert_fp32_within_ulps

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def case(msg):
    print(f"[case] {msg}", flush=True)


@pytest.mark.parametrize("N,K,w_bits", [(8, 16, 8), (300, 1040, 8), (129, 768, 6), (64, 4096, 4),
                                        (33, 5120, 3)])
def test_fold_asym_bit_exact(N, K, w_bits):
    case(f"fold_asym N={N} K={K} w_bits={w_bits}")
    r = np.random.default_rng(N * 3 + K)
    W = (r.standard_normal((N, K)) * 0.02 + r.uniform(-0.03, 0.03, (N, 1))).astype(np.float16)
    W[0] = 0.0                          # zero row
    W[1] = np.abs(W[1])                 # one-sided rows: zero point at an end
    W[2] = -np.abs(W[2])
    b = r.normal(0, 0.02, N).astype(np.float16)
    z = r.normal(0, 1, K).astype(np.float32)
    s = r.uniform(0.05, 2.0, K).astype(np.float32)
    Wq, sW, zW, bp = ot.fold_weights_asym(dev(W), dev(b), w_bits, dev(z), dev(s))
    rW, rs, rz, rb = O.fold_weights_asym(W, b, z, s, w_bits)
    assert np.array_equal(host(sW).view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(host(zW), rz)
    assert np.array_equal(host(Wq), rW)
    assert_fp32_within_ulps(host(bp), rb, 1)


def test_fold_asym_rejects_non_finite():
    W = torch.zeros((4, 32), dtype=torch.float16, device="cuda")
    W[1, 3] = float("inf")
    one = torch.ones(32, device="cuda")
    with pytest.raises(ot.OTError):
        ot.fold_weights_asym(W, None, 8, torch.zeros(32, device="cuda"), one)


ASYM_SHAPES = [(1, 8, 16), (5, 772, 768), (17, 100, 400), (33, 64, 48), (64, 1000, 2064),
               (48, 8193, 96), (20, 16448, 528), (64, 33000, 272),
               (65, 256, 128), (300, 772, 1040), (513, 129, 768), (600, 1024, 4112)]


@pytest.mark.parametrize("M,N,K", ASYM_SHAPES)
def test_qlinear_asym_parity(M, N, K):
    case(f"qlinear_asym M={M} N={N} K={K}")
    r = np.random.default_rng(M * 1000 + N + K)
    Xq = r.integers(-127, 128, size=(M, K)).astype(np.int8)
    Wq = r.integers(-128, 128, size=(N, K)).astype(np.int8)
    zW = r.integers(-128, 128, size=N).astype(np.int32)
    sW = (r.uniform(0.5, 2.0, N) * 1e-3).astype(np.float32)
    bp = r.normal(0, 1, N).astype(np.float32)
    Y, acc = ot.qlinear_asym(dev(Xq), dev(Wq), dev(sW), dev(zW), dev(bp), 8, 8, want_acc=True)
    Y2 = ot.qlinear_asym(dev(Xq), dev(Wq), dev(sW), dev(zW), dev(bp), 8, 8)
    racc = O.int_gemm_asym(Xq, Wq, zW)
    assert np.array_equal(host(acc), racc)
    rY = O.epilogue(racc, sW, bp)
    assert_fp16_close(host(Y), rY)
    assert_fp16_close(host(Y2), rY)


def test_qlinear_asym_extreme_codes_near_the_limit():
    """Largest K the ABI allows at W8A8 (K * 127 * 256 < 2^31) with every
    code at its extreme: the row sums and the zero-point product are exact."""
    K, N = 66048, 40
    for M in (3, 80):
        case(f"qlinear_asym extreme M={M} K={K}")
        Xq = np.full((M, K), -127, dtype=np.int8)
        Xq[0] = 127
        Wq = np.full((N, K), 127, dtype=np.int8)
        Wq[1] = -128
        zW = np.full(N, -128, dtype=np.int32)
        zW[1] = 127
        sW = np.full(N, 1e-9, dtype=np.float32)
        bp = np.zeros(N, dtype=np.float32)
        _, acc = ot.qlinear_asym(dev(Xq), dev(Wq), dev(sW), dev(zW), dev(bp), 8, 8, want_acc=True)
        assert np.array_equal(host(acc), O.int_gemm_asym(Xq, Wq, zW))


@pytest.mark.parametrize("name,li,M", [("opt125m_w8a8", 0, 16), ("opt13b_w6a6", 0, 300),
                                       ("opt30b_decode_w8a8", 2, 8)])
def test_asym_pipeline_on_workload_layers(name, li, M):
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    case(f"asym pipeline {name}/{lay.name} M={M}")
    batches = list(synth.calibration_batches(wl, li, 64, 2))
    X = synth.activations(wl, li, M)
    W = synth.weight(wl, li)
    b = synth.bias(wl, li)
    _, z, s, inv_s = ot.calibrate(batches, wl.a_bits)
    Wq, sW, zW, bp = ot.fold_weights_asym(dev(W), dev(b), wl.w_bits, z, s)
    Xq = ot.quantize_act(dev(X), wl.a_bits, z, inv_s)
    Y, acc = ot.qlinear_asym(Xq, Wq, sW, zW, bp, wl.a_bits, wl.w_bits, want_acc=True)
    _, rz, rs, rinv = O.calibrate(batches, wl.a_bits)
    rW, rsW, rzW, rb = O.fold_weights_asym(W, b, rz, rs, wl.w_bits)
    rq = O.quantize_act(X, rz, rinv, wl.a_bits)
    assert np.array_equal(host(Wq), rW) and np.array_equal(host(zW), rzW)
    racc = O.int_gemm_asym(rq, rW, rzW)
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), O.epilogue(racc, rsW, rb))

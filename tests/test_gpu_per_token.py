"""GPU parity of the per-token path (Eq. (c) and (h): ot_quantize_act_per_token,
ot_fold_weights_per_token, ot_qlinear_per_token) against the CPU oracle,
through the C ABI.  Codes, scales, accumulators and b' are bit-exact; the
fp16 output is within 2 fp16 ulp and 1e-3 relative error."""
import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import ot, synth
from tests._tol import assert_fp16_close

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def case(msg):
    print(f"[case] {msg}", flush=True)


def _acts(M, K, seed):
    r = np.random.default_rng(seed)
    X = r.standard_normal((M, K)) * r.uniform(0.01, 30, (M, 1))
    X[:, r.choice(K, max(1, K // 200), replace=False)] *= 20
    if M > 2:
        X[1] = 0.0  # a zero row takes scale 1
    return np.clip(X, -65504, 65504).astype(np.float16)


@pytest.mark.parametrize("M,K", [(1, 16), (3, 768), (17, 1040), (130, 512), (64, 4096),
                                 (9, 5120), (5, 16384), (2, 16400), (3, 32768), (1, 65536)])
@pytest.mark.parametrize("a_bits", [8, 6])
def test_quantize_per_token_bit_exact(M, K, a_bits):
    case(f"quantize_per_token M={M} K={K} a_bits={a_bits}")
    X = _acts(M, K, M * 7 + K + a_bits)
    Xq, sX = ot.quantize_act_per_token(dev(X), a_bits)
    rq, rs = O.quantize_act_per_token(X, a_bits)
    assert np.array_equal(host(sX).view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(host(Xq), rq)


@pytest.mark.parametrize("N,K,w_bits", [(8, 16, 8), (300, 1040, 8), (129, 768, 6), (64, 4096, 4)])
def test_fold_per_token_bit_exact(N, K, w_bits):
    case(f"fold_per_token N={N} K={K} w_bits={w_bits}")
    r = np.random.default_rng(N + K)
    W = (r.standard_normal((N, K)) * 0.02).astype(np.float16)
    W[0] = 0.0  # zero row -> sW = 1
    b = r.normal(0, 0.02, N).astype(np.float16)
    zres = r.normal(0, 2, N).astype(np.float32)
    for bb, zz in ((b, zres), (None, None), (b, None), (None, zres)):
        Wq, sW, bp = ot.fold_weights_per_token(dev(W), None if bb is None else dev(bb),
                                               None if zz is None else dev(zz), w_bits)
        rW, rs, rb = O.fold_weights_per_token(W, bb, zz, w_bits)
        assert np.array_equal(host(Wq), rW)
        assert np.array_equal(host(sW).view(np.uint32), rs.view(np.uint32))
        assert np.array_equal(host(bp).view(np.uint32), rb.view(np.uint32))


def test_fold_per_token_rejects_non_finite():
    W = torch.zeros((4, 32), dtype=torch.float16, device="cuda")
    zres = torch.tensor([0.0, float("inf"), 0.0, 0.0], device="cuda")
    with pytest.raises(ot.OTError):
        ot.fold_weights_per_token(W, None, zres, 8)
    W[2, 5] = float("nan")
    with pytest.raises(ot.OTError):
        ot.fold_weights_per_token(W, None, None, 8)


# decode (M <= 64, every tile height) and prefill tiles, ragged N and K
PT_SHAPES = [(1, 8, 16), (5, 772, 768), (17, 100, 400), (33, 64, 48), (64, 1000, 2064),
             (48, 8193, 96), (20, 16448, 528), (64, 33000, 272),
             (65, 256, 128), (300, 772, 1040), (513, 129, 768), (600, 1024, 4112)]


@pytest.mark.parametrize("M,N,K", PT_SHAPES)
def test_qlinear_per_token_parity(M, N, K):
    case(f"qlinear_per_token M={M} N={N} K={K}")
    r = np.random.default_rng(M * 1000 + N + K)
    Xq = r.integers(-127, 128, size=(M, K)).astype(np.int8)
    Wq = r.integers(-127, 128, size=(N, K)).astype(np.int8)
    sX = (r.uniform(0.5, 2.0, M) * 1e-2).astype(np.float32)
    sW = (r.uniform(0.5, 2.0, N) * 1e-3).astype(np.float32)
    bp = r.normal(0, 1, N).astype(np.float32)
    Y, acc = ot.qlinear_per_token(dev(Xq), dev(Wq), dev(sX), dev(sW), dev(bp), 8, 8, want_acc=True)
    Y2 = ot.qlinear_per_token(dev(Xq), dev(Wq), dev(sX), dev(sW), dev(bp), 8, 8)
    racc = O.int_gemm(Xq, Wq)
    assert np.array_equal(host(acc), racc)
    rY = O.epilogue_per_token(racc, sX, sW, bp)
    assert_fp16_close(host(Y), rY)
    assert_fp16_close(host(Y2), rY)


@pytest.mark.parametrize("name,li,M", [("opt13b_w6a6", 1, 300), ("opt13b_w6a6", 3, 64),
                                       ("opt6.7b_w8a8", 3, 129), ("opt30b_decode_w8a8", 1, 8)])
def test_per_token_pipeline_on_workload_layers(name, li, M):
    """out / fc2 shapes through the whole per-token path, with a symmetrized
    residual shift zres carried into the bias."""
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    case(f"per-token pipeline {name}/{lay.name} M={M}")
    X = synth.activations(wl, li, M)
    W = synth.weight(wl, li)
    b = synth.bias(wl, li)
    zres = np.random.default_rng(li).normal(0, 1, lay.N).astype(np.float32)
    Xq, sX = ot.quantize_act_per_token(dev(X), wl.a_bits)
    Wq, sW, bp = ot.fold_weights_per_token(dev(W), dev(b), dev(zres), wl.w_bits)
    Y, acc = ot.qlinear_per_token(Xq, Wq, sX, sW, bp, wl.a_bits, wl.w_bits, want_acc=True)
    rq, rs = O.quantize_act_per_token(X, wl.a_bits)
    rW, rsW, rb = O.fold_weights_per_token(W, b, zres, wl.w_bits)
    assert np.array_equal(host(Xq), rq) and np.array_equal(host(Wq), rW)
    racc = O.int_gemm(rq, rW)
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), O.epilogue_per_token(racc, rs, rsW, rb))


def test_per_token_rejects_overflowing_k_and_bad_pointers():
    Xq = torch.zeros((2, 133152), dtype=torch.int8, device="cuda")
    Wq = torch.zeros((4, 133152), dtype=torch.int8, device="cuda")
    f = torch.zeros(4, device="cuda")
    with pytest.raises(ot.OTError):
        ot.qlinear_per_token(Xq, Wq, f[:2].contiguous(), f, f, 8, 8)
    x = torch.zeros((2, 65536 + 16), dtype=torch.float16, device="cuda")
    with pytest.raises(ot.OTError):
        ot.quantize_act_per_token(x, 8)

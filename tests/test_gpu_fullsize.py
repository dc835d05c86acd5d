"""Full-size parity: every linear of the OPT-6.7B, OPT-13B, OPT-30B (decode)
and OPT-66B workloads at their real shapes, through the C ABI, in the launch
configuration bench.py times (no acc_out for Y), against the oracle, on
every element.

Calibration (minmax, z, s, 1/s) is compared on every channel; the weight
fold (Wq, sW, b') on every output channel; the activation codes on every
token; the int32 accumulators (through acc_out) and the fp16 outputs on
every token x channel.  The oracle's fold and integer GEMM run in chunks of
output channels so that host memory stays bounded; each chunk is exact, so
chunking changes nothing.
"""
import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import ot, synth
from tests._tol import assert_fp16_close, assert_fp32_within_ulps

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

PREFILL = [("opt6.7b_w8a8", i) for i in range(4)] + [("opt13b_w6a6", i) for i in range(4)] + \
          [("opt66b_w8a8", i) for i in range(4)]
DECODE = [("opt30b_decode_w8a8", i) for i in range(4)]
# output channels per oracle chunk: its float64 product [M x chunk] stays
# within about 1 GB
CHUNK_BYTES = 1 << 30


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ot.lib()
    yield
    torch.cuda.synchronize()


def _prepare(wl, li, rows):
    """GPU path for one layer; returns host copies of what is compared."""
    lay = wl.layers[li]
    batches = list(synth.calibration_batches(wl, li))
    W = synth.weight(wl, li)
    b = synth.bias(wl, li)
    X = synth.activations(wl, li, rows)
    minmax, z, s, inv_s = ot.calibrate(batches, wl.a_bits)
    Wq, sW, bp = ot.fold_weights(torch.from_numpy(W).cuda(), torch.from_numpy(b).cuda(),
                                 wl.w_bits, z, s)
    Xq = ot.quantize_act(torch.from_numpy(X).cuda(), wl.a_bits, z, inv_s)
    torch.cuda.synchronize()
    qa, qw = O.qmax(wl.a_bits), O.qmax(wl.w_bits)
    assert int(Xq.abs().max()) <= qa and int(Wq.abs().max()) <= qw
    return dict(batches=batches, W=W, b=b, X=X, minmax=minmax.cpu().numpy(), z=z.cpu().numpy(),
                s=s.cpu().numpy(), inv_s=inv_s.cpu().numpy(), Wq_dev=Wq, sW_dev=sW, bp_dev=bp,
                Xq_dev=Xq, K=lay.K, N=lay.N)


def _check_calibration(wl, g):
    ref = O.calibrate(g["batches"], wl.a_bits)
    for got, r, name in zip((g["minmax"], g["z"], g["s"], g["inv_s"]), ref,
                            ("minmax", "z", "s", "inv_s")):
        assert np.array_equal(got.view(np.uint32), r.view(np.uint32)), name
    return ref


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,li", PREFILL)
def test_prefill_layer_every_element(name, li):
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    M, N, K = wl.M, lay.N, lay.K
    print(f"[case] fullsize {name}/{lay.name} M={M} K={K} N={N} "
          f"kernel={ot.ot_qlinear_plan(M, N, K)}", flush=True)
    g = _prepare(wl, li, M)
    _, z, s, inv_s = _check_calibration(wl, g)
    # the launch bench.py times (no accumulator output), then the test path
    Y = ot.qlinear(g["Xq_dev"], g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits, wl.w_bits)
    Y2, acc = ot.qlinear(g["Xq_dev"], g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits,
                         wl.w_bits, want_acc=True)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2)
    del Y2
    # every token's codes
    rXq = O.quantize_act(g["X"], z, inv_s, wl.a_bits)
    assert np.array_equal(g["Xq_dev"].cpu().numpy(), rXq)
    O.check_acc_range(K, wl.a_bits, wl.w_bits)
    chunk = max(256, CHUNK_BYTES // (8 * M) // 256 * 256)
    for n0 in range(0, N, chunk):
        n1 = min(N, n0 + chunk)
        rWq, rsW, rbp = O.fold_weights(g["W"][n0:n1], g["b"][n0:n1], z, s, wl.w_bits)
        assert np.array_equal(g["Wq_dev"][n0:n1].cpu().numpy(), rWq), f"Wq [{n0}, {n1})"
        assert np.array_equal(g["sW_dev"][n0:n1].cpu().numpy().view(np.uint32),
                              rsW.view(np.uint32)), f"sW [{n0}, {n1})"
        assert_fp32_within_ulps(g["bp_dev"][n0:n1].cpu().numpy(), rbp, 1)
        racc = O.int_gemm(rXq, rWq)
        assert np.array_equal(acc[:, n0:n1].cpu().numpy(), racc), f"acc [{n0}, {n1})"
        assert_fp16_close(Y[:, n0:n1].cpu().numpy(), O.epilogue(racc, rsW, rbp),
                          f"Y [{n0}, {n1})")
        del racc
        print(f"  channels [{n0}, {n1}) of {N} match", flush=True)


@pytest.mark.parametrize("name,li", DECODE)
def test_decode_layer_full(name, li):
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    Mmax = max(wl.decode_M)
    print(f"[case] fullsize {name}/{lay.name} M<={Mmax} K={lay.K} N={lay.N}", flush=True)
    g = _prepare(wl, li, Mmax)
    _, z, s, inv_s = _check_calibration(wl, g)
    # the oracle folds every channel itself (decode layers are small enough)
    rWq, rsW, rbp = O.fold_weights(g["W"], g["b"], z, s, wl.w_bits)
    assert np.array_equal(g["Wq_dev"].cpu().numpy(), rWq)
    assert np.array_equal(g["sW_dev"].cpu().numpy().view(np.uint32), rsW.view(np.uint32))
    assert_fp32_within_ulps(g["bp_dev"].cpu().numpy(), rbp, 1)
    rXq = O.quantize_act(g["X"], z, inv_s, wl.a_bits)
    assert np.array_equal(g["Xq_dev"].cpu().numpy(), rXq)
    racc = O.int_gemm(rXq, rWq)  # all 64 tokens x all channels
    rY = O.epilogue(racc, rsW, rbp)
    Wp = ot.pack_weights(g["Wq_dev"])
    for M in wl.decode_M:
        Xm = g["Xq_dev"][:M].contiguous()
        Y = ot.qlinear(Xm, g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits, wl.w_bits)
        Y2, acc = ot.qlinear(Xm, g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits, wl.w_bits,
                             want_acc=True)
        # the benchmark's launches: a workspace (split K where the plan takes
        # it), on row-major and on packed weights
        Y3, acc3 = ot.qlinear(Xm, g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits, wl.w_bits,
                              want_acc=True, workspace=True)
        Y4, acc4 = ot.qlinear_packed(Xm, Wp, lay.N, g["sW_dev"], g["bp_dev"], wl.a_bits,
                                     wl.w_bits, want_acc=True, workspace=True)
        torch.cuda.synchronize()
        assert np.array_equal(acc.cpu().numpy(), racc[:M]), f"acc M={M}"
        assert np.array_equal(acc3.cpu().numpy(), racc[:M]), f"acc (workspace) M={M}"
        assert np.array_equal(acc4.cpu().numpy(), racc[:M]), f"acc (packed) M={M}"
        assert_fp16_close(Y.cpu().numpy(), rY[:M], f"Y M={M}")
        assert_fp16_close(Y2.cpu().numpy(), rY[:M], f"Y(acc path) M={M}")
        assert torch.equal(Y3, Y) and torch.equal(Y4, Y), f"Y (workspace, packed) M={M}"


# The two other epilogue flavours at full size, on the OPT-13B W6A6 layers
# (4096 tokens, every element): asymmetric ("Int8") weights, Eq. (a), on
# all four linears, and the paper's per-token path, Eq. (c), on the two it
# applies to (out and fc2), as the benchmark's asym_weights and mixed_block
# steps run them.
OPT13B = [("opt13b_w6a6", i) for i in range(4)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,li", OPT13B)
def test_prefill_asym_layer_every_element(name, li):
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    M, N, K = wl.M, lay.N, lay.K
    print(f"[case] fullsize asymmetric {name}/{lay.name} M={M} K={K} N={N} "
          f"kernel={ot.ot_qlinear_plan(M, N, K)}", flush=True)
    g = _prepare(wl, li, M)
    _, z, s, inv_s = _check_calibration(wl, g)
    Wq, sW, zW, bp = ot.fold_weights_asym(torch.from_numpy(g["W"]).cuda(),
                                          torch.from_numpy(g["b"]).cuda(), wl.w_bits,
                                          torch.from_numpy(z).cuda(), torch.from_numpy(s).cuda())
    Y = ot.qlinear_asym(g["Xq_dev"], Wq, sW, zW, bp, wl.a_bits, wl.w_bits)
    Y2, acc = ot.qlinear_asym(g["Xq_dev"], Wq, sW, zW, bp, wl.a_bits, wl.w_bits, want_acc=True)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2)
    del Y2
    rXq = O.quantize_act(g["X"], z, inv_s, wl.a_bits)
    assert np.array_equal(g["Xq_dev"].cpu().numpy(), rXq)
    chunk = max(256, CHUNK_BYTES // (8 * M) // 256 * 256)
    for n0 in range(0, N, chunk):
        n1 = min(N, n0 + chunk)
        rWq, rsW, rzW, rbp = O.fold_weights_asym(g["W"][n0:n1], g["b"][n0:n1], z, s, wl.w_bits)
        assert np.array_equal(Wq[n0:n1].cpu().numpy(), rWq), f"Wq [{n0}, {n1})"
        assert np.array_equal(sW[n0:n1].cpu().numpy().view(np.uint32), rsW.view(np.uint32))
        assert np.array_equal(zW[n0:n1].cpu().numpy(), rzW), f"zW [{n0}, {n1})"
        assert_fp32_within_ulps(bp[n0:n1].cpu().numpy(), rbp, 1)
        racc = O.int_gemm_asym(rXq, rWq, rzW)
        assert np.array_equal(acc[:, n0:n1].cpu().numpy(), racc), f"acc [{n0}, {n1})"
        assert_fp16_close(Y[:, n0:n1].cpu().numpy(), O.epilogue(racc, rsW, rbp),
                          f"Y [{n0}, {n1})")
        del racc
        print(f"  channels [{n0}, {n1}) of {N} match", flush=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,li", [("opt13b_w6a6", 1), ("opt13b_w6a6", 3)])
def test_prefill_per_token_layer_every_element(name, li):
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    M, N, K = wl.M, lay.N, lay.K
    print(f"[case] fullsize per-token {name}/{lay.name} M={M} K={K} N={N} "
          f"kernel={ot.ot_qlinear_plan(M, N, K)}", flush=True)
    W = synth.weight(wl, li)
    b = synth.bias(wl, li)
    X = synth.activations(wl, li, M)
    Xq, sX = ot.quantize_act_per_token(torch.from_numpy(X).cuda(), wl.a_bits)
    Wq, sW, bp = ot.fold_weights_per_token(torch.from_numpy(W).cuda(), torch.from_numpy(b).cuda(),
                                           None, wl.w_bits)
    Y = ot.qlinear_per_token(Xq, Wq, sX, sW, bp, wl.a_bits, wl.w_bits)
    Y2, acc = ot.qlinear_per_token(Xq, Wq, sX, sW, bp, wl.a_bits, wl.w_bits, want_acc=True)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2)
    del Y2
    rXq, rsX = O.quantize_act_per_token(X, wl.a_bits)
    assert np.array_equal(Xq.cpu().numpy(), rXq)
    assert np.array_equal(sX.cpu().numpy().view(np.uint32), rsX.view(np.uint32))
    chunk = max(256, CHUNK_BYTES // (8 * M) // 256 * 256)
    for n0 in range(0, N, chunk):
        n1 = min(N, n0 + chunk)
        rWq, rsW, rbp = O.fold_weights_per_token(W[n0:n1], b[n0:n1], None, wl.w_bits)
        assert np.array_equal(Wq[n0:n1].cpu().numpy(), rWq), f"Wq [{n0}, {n1})"
        assert np.array_equal(sW[n0:n1].cpu().numpy().view(np.uint32), rsW.view(np.uint32))
        assert_fp32_within_ulps(bp[n0:n1].cpu().numpy(), rbp, 1)
        racc = O.int_gemm(rXq, rWq)
        assert np.array_equal(acc[:, n0:n1].cpu().numpy(), racc), f"acc [{n0}, {n1})"
        assert_fp16_close(Y[:, n0:n1].cpu().numpy(), O.epilogue_per_token(racc, rsX, rsW, rbp),
                          f"Y [{n0}, {n1})")
        del racc
        print(f"  channels [{n0}, {n1}) of {N} match", flush=True)

"""Full-size parity: every linear of the OPT-6.7B, OPT-13B, OPT-30B (decode)
and OPT-66B workloads at their real shapes, through the C ABI, in the launch
configuration bench.py times (no acc_out for Y), against the oracle.

Calibration, z, s and 1/s are compared on every channel; for prefill layers
the weight fold on sampled output channels, and codes, accumulators and
outputs on sampled tokens x sampled channels (the oracle computes those one
by one); for decode layers the oracle folds every channel.  Properties that
hold at any size (code ranges) are checked on every element.  Decode shapes
(at most 64 tokens) are compared on every output.
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
N_TOKENS = 48
N_CHANNELS = 192


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ot.lib()
    yield
    torch.cuda.synchronize()


def _sample(n, k, seed):
    r = np.random.default_rng(seed)
    idx = set(r.choice(n, size=min(k, n), replace=False).tolist()) | {0, n - 1}
    return np.array(sorted(idx))


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


@pytest.mark.parametrize("name,li", PREFILL)
def test_prefill_layer_sampled(name, li):
    wl = synth.WORKLOADS[name]
    lay = wl.layers[li]
    print(f"[case] fullsize {name}/{lay.name} M={wl.M} K={lay.K} N={lay.N}", flush=True)
    g = _prepare(wl, li, wl.M)
    _, z, s, inv_s = _check_calibration(wl, g)
    m_idx = _sample(wl.M, N_TOKENS, 1 + li)
    n_idx = _sample(lay.N, N_CHANNELS, 2 + li)
    # the launch bench.py times (no accumulator output), then the test path
    Y = ot.qlinear(g["Xq_dev"], g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits, wl.w_bits)
    Y2, acc = ot.qlinear(g["Xq_dev"], g["Wq_dev"], g["sW_dev"], g["bp_dev"], wl.a_bits,
                         wl.w_bits, want_acc=True)
    torch.cuda.synchronize()
    mi = torch.from_numpy(m_idx).cuda()
    ni = torch.from_numpy(n_idx).cuda()
    Ys = Y.index_select(0, mi).index_select(1, ni).cpu().numpy()
    Y2s = Y2.index_select(0, mi).index_select(1, ni).cpu().numpy()
    accs = acc.index_select(0, mi).index_select(1, ni).cpu().numpy()
    Xq_s = g["Xq_dev"].index_select(0, mi).cpu().numpy()
    Wq_s = g["Wq_dev"].index_select(0, ni).cpu().numpy()
    sW_s = g["sW_dev"].index_select(0, ni).cpu().numpy()
    bp_s = g["bp_dev"].index_select(0, ni).cpu().numpy()
    del Y, Y2, acc
    # oracle on the samples
    rWq, rsW, rbp = O.fold_weights(g["W"][n_idx], g["b"][n_idx], z, s, wl.w_bits)
    assert np.array_equal(Wq_s, rWq)
    assert np.array_equal(sW_s.view(np.uint32), rsW.view(np.uint32))
    assert_fp32_within_ulps(bp_s, rbp, 1)
    rXq = O.quantize_act(g["X"][m_idx], z, inv_s, wl.a_bits)
    assert np.array_equal(Xq_s, rXq)
    racc = O.int_gemm(rXq, rWq)
    assert np.array_equal(accs, racc)
    rY = O.epilogue(racc, rsW, rbp)
    assert_fp16_close(Ys, rY)
    assert_fp16_close(Y2s, rY)


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

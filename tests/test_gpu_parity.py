"""Parity of libot (through its C ABI) with the CPU oracle, element by element.

Integer stages (minmax, z, s, inv_s, Wq, sW, Xq, acc) must be bit-exact; the
compensated bias within 1 fp32 ulp (its fp64 sum order is unspecified); the
fp16 output within 2 fp16 ulp and 1e-3 relative error.
"""
import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import ot, synth
from tests._tol import assert_fp16_close, assert_fp32_within_ulps

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ot.lib()
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def case(msg):
    print(f"[case] {msg}", flush=True)


# --------------------------------------------------------------------------
# Calibration
# --------------------------------------------------------------------------
@pytest.mark.parametrize("a_bits", [8, 6, 3])
def test_calibrate_streamed_batches_bit_exact(a_bits):
    wl = synth.WORKLOADS["opt125m_w8a8"]
    batches = list(synth.calibration_batches(wl, 0))
    case(f"calibrate opt125m a_bits={a_bits}")
    got = [host(t) for t in ot.calibrate(batches, a_bits)]
    ref = O.calibrate(batches, a_bits)
    for g, r, name in zip(got, ref, ["minmax", "z", "s", "inv_s"]):
        assert np.array_equal(g.view(np.uint32), r.view(np.uint32)), name


def test_calibrate_ragged_and_special_values():
    r = np.random.default_rng(7)
    K = 37  # not a multiple of anything the kernels tile by
    a = r.normal(0, 3, size=(131, K)).astype(np.float16)
    a[:, 0] = 2.0                  # constant channel -> s = 1
    a[:, 1] = -0.0                 # all negative zeros -> +0
    a[5, 2] = np.float16(65504)    # fp16 extremes
    a[6, 2] = np.float16(-65504)
    b = r.normal(1, 1, size=(3, K)).astype(np.float16)
    case("calibrate ragged K=37")
    got = [host(t) for t in ot.calibrate([a, b], 8)]
    ref = O.calibrate([a, b], 8)
    for g, rr, name in zip(got, ref, ["minmax", "z", "s", "inv_s"]):
        assert np.array_equal(g.view(np.uint32), rr.view(np.uint32)), name


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_calibrate_rejects_non_finite_then_recovers(bad):
    x = np.ones((8, 32), dtype=np.float16)
    x[3, 5] = bad
    K = 32
    minmax = torch.empty(2 * K, dtype=torch.float32, device="cuda")
    z, s, inv_s = (torch.full((K,), 7.0, device="cuda") for _ in range(3))
    case(f"calibrate non-finite {bad}")
    with pytest.raises(ot.OTError) as e:
        ot.ot_calibrate(dev(x), 8, True, minmax, z, s, inv_s)
    assert e.value.code == ot.OT_ENONFINITE
    assert torch.all(z == 7.0)  # outputs untouched
    good = np.ones((8, 32), dtype=np.float16)
    ot.ot_calibrate(dev(good), 8, True, minmax, z, s, inv_s)
    assert torch.all(z == 1.0) and torch.all(s == 1.0)


# --------------------------------------------------------------------------
# Weight fold
# --------------------------------------------------------------------------
@pytest.mark.parametrize("w_bits,with_bias", [(8, True), (6, True), (4, False)])
def test_fold_weights_parity(w_bits, with_bias):
    wl = synth.WORKLOADS["opt125m_w8a8"]
    _, z, s, _ = O.calibrate(list(synth.calibration_batches(wl, 0)), 8)
    W = synth.weight(wl, 0).copy()
    W[3] = 0  # an all-zero row
    b = synth.bias(wl, 0) if with_bias else None
    case(f"fold opt125m w_bits={w_bits} bias={with_bias}")
    Wq, sW, bp = ot.fold_weights(dev(W), None if b is None else dev(b), w_bits, dev(z), dev(s))
    rWq, rsW, rbp = O.fold_weights(W, b, z, s, w_bits)
    assert np.array_equal(host(Wq), rWq)
    assert np.array_equal(host(sW).view(np.uint32), rsW.view(np.uint32))
    assert_fp32_within_ulps(host(bp), rbp, 1)


def test_fold_rejects_non_finite():
    W = np.ones((4, 32), dtype=np.float16)
    W[2, 7] = np.inf
    case("fold non-finite")
    with pytest.raises(ot.OTError) as e:
        ot.fold_weights(dev(W), None, 8, dev(np.zeros(32, np.float32)), dev(np.ones(32, np.float32)))
    assert e.value.code == ot.OT_ENONFINITE
    b = np.array([0, np.nan, 0, 0], dtype=np.float16)
    with pytest.raises(ot.OTError):
        ot.fold_weights(dev(np.ones((4, 32), np.float16)), dev(b), 8,
                        dev(np.zeros(32, np.float32)), dev(np.ones(32, np.float32)))


# --------------------------------------------------------------------------
# Activation quantization
# --------------------------------------------------------------------------
@pytest.mark.parametrize("M,K,a_bits", [(16, 768, 8), (1, 16, 8), (3, 48, 6), (33, 1040, 8),
                                        (70, 2064, 4), (257, 5120, 6)])
def test_quantize_act_parity(M, K, a_bits):
    r = np.random.default_rng(M * 7 + K)
    x = (r.standard_normal((M, K)) * r.uniform(0.5, 30, size=K) + r.uniform(-5, 5, size=K))
    x = x.astype(np.float16)
    _, z, s, inv_s = O.calibrate([x[: max(1, M // 2)]], a_bits)  # later rows go out of range
    case(f"quantize M={M} K={K} a_bits={a_bits}")
    got = host(ot.quantize_act(dev(x), a_bits, dev(z), dev(inv_s)))
    assert np.array_equal(got, O.quantize_act(x, z, inv_s, a_bits))


def test_quantize_act_rows_beyond_one_grid():
    # more rows than one launch grid covers (65535 x 16 row groups of 4 rows
    # per wave, 4 waves per workgroup): the waves loop over further groups,
    # and the last group is ragged
    M, K = 65535 * 16 + 37, 32
    r = np.random.default_rng(11)
    x = (r.standard_normal((M, K)) * 3).astype(np.float16)
    z = r.uniform(-1, 1, size=K).astype(np.float32)
    inv_s = r.uniform(2, 20, size=K).astype(np.float32)
    case(f"quantize grid-stride M={M} K={K}")
    got = host(ot.quantize_act(dev(x), 8, dev(z), dev(inv_s)))
    assert np.array_equal(got, O.quantize_act(x, z, inv_s, 8))


def test_quantize_act_ties_and_clamps():
    v = np.array([2.5, 3.5, -2.5, -0.5, 0.5, 1.5, 200.0, -200.0, 126.5, -127.5, 0.0, -0.0,
                  65504, -65504, 1e-7, 6.5], dtype=np.float16)
    x = np.tile(v, (2, 1))
    K = x.shape[1]
    z = np.zeros(K, np.float32)
    one = np.ones(K, np.float32)
    case("quantize ties")
    got = host(ot.quantize_act(dev(x), 8, dev(z), dev(one)))
    assert np.array_equal(got, O.quantize_act(x, z, one, 8))


# --------------------------------------------------------------------------
# Quantized linear on random codes: every tile shape, ragged edges
# --------------------------------------------------------------------------
def _random_qlinear_inputs(M, N, K, a_bits, w_bits, seed):
    r = np.random.default_rng(seed)
    qa, qw = O.qmax(a_bits), O.qmax(w_bits)
    Xq = r.integers(-qa, qa + 1, size=(M, K)).astype(np.int8)
    Wq = r.integers(-qw, qw + 1, size=(N, K)).astype(np.int8)
    sW = (r.uniform(0.5, 2.0, size=N) * 1e-3).astype(np.float32)
    bp = r.normal(0, 1, size=N).astype(np.float32)
    return Xq, Wq, sW, bp


QL_SHAPES = [
    # decode kernel (M <= 64)
    (1, 8, 16), (1, 300, 1040), (5, 772, 768), (16, 256, 4096), (17, 100, 400),
    (32, 513, 128), (33, 64, 48), (64, 1000, 2064),
    # decode kernel, every tile for up to 16 tokens (16-row tiles up to
    # N = 4096, 32-row tiles with 512-byte K slices up to 8192, 32-row tiles
    # with 128-byte slices beyond) and, for 17-32 and 33-64 tokens, every
    # tile height the unsplit launch plan picks (32, 64, 96 and 128 rows
    # while a grid fits one pass over 256 CUs, 64 rows beyond), on both sides
    # of the one-pass boundaries, with ragged N and K tails
    (1, 4096, 528), (2, 4097, 1040), (3, 7168, 1040), (16, 5000, 2064), (8, 8192, 48),
    (1, 16400, 272), (9, 16384, 2064), (20, 16448, 528), (64, 16392, 784),
    (32, 8192, 512), (48, 8193, 96), (17, 8195, 2000), (33, 12000, 1040),
    (24, 32768, 160), (40, 32769, 64), (64, 33000, 272), (18, 40003, 48),
    (48, 20000, 1040), (30, 20000, 528), (64, 24576, 272), (17, 24577, 1040),
    (40, 30000, 1040),
    # prefill kernel; half the tiles (a checkerboard) walk K from its second
    # 128-byte tile and wrap round: grids with such tiles at one K tile
    # (K = 48, 128) and at two with a ragged tail (K = 144)
    (65, 256, 128), (200, 300, 400), (256, 256, 256), (300, 772, 1040), (513, 129, 768),
    (600, 1024, 4112), (300, 772, 48), (257, 600, 128), (520, 700, 144),
]


@pytest.mark.parametrize("M,N,K", QL_SHAPES)
def test_qlinear_parity_random_codes(M, N, K):
    Xq, Wq, sW, bp = _random_qlinear_inputs(M, N, K, 8, 8, M * 1000 + N + K)
    case(f"qlinear M={M} N={N} K={K}")
    Y, acc = ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8, want_acc=True)
    racc = O.int_gemm(Xq, Wq)
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), O.epilogue(racc, sW, bp))


@pytest.mark.parametrize("M", [7, 64, 300])
def test_qlinear_extreme_codes_near_int32_limit(M):
    # K * 127 * 127 just below 2^31: the largest accumulators the ABI allows
    K, N = 133136, 48
    Xq = np.full((M, K), 127, dtype=np.int8)
    Xq[1::2] = -127
    Wq = np.full((N, K), 127, dtype=np.int8)
    Wq[::3, ::2] = -127
    sW = np.full(N, 1e-6, dtype=np.float32)
    bp = np.zeros(N, dtype=np.float32)
    case(f"qlinear extreme M={M} K={K}")
    Y, acc = ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8, want_acc=True)
    racc = O.int_gemm(Xq, Wq)
    assert np.abs(racc.astype(np.int64)).max() == K * 127 * 127
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), O.epilogue(racc, sW, bp))


def test_qlinear_output_overflow_is_inf():
    M, N, K = 4, 8, 64
    Xq = np.full((M, K), 127, dtype=np.int8)
    Wq = np.full((N, K), 127, dtype=np.int8)
    sW = np.full(N, 1.0, dtype=np.float32)  # 64 * 127^2 = 1032256 > 65504
    bp = np.zeros(N, dtype=np.float32)
    Y = host(ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8))
    assert np.all(np.isposinf(Y))


def test_qlinear_rejects_overflowing_k():
    Xq = torch.zeros((2, 133152), dtype=torch.int8, device="cuda")
    Wq = torch.zeros((4, 133152), dtype=torch.int8, device="cuda")
    with pytest.raises(ot.OTError) as e:
        ot.qlinear(Xq, Wq, torch.ones(4, device="cuda"), torch.zeros(4, device="cuda"), 8, 8)
    assert e.value.code == ot.OT_ERANGE


def test_qlinear_is_deterministic():
    Xq, Wq, sW, bp = _random_qlinear_inputs(512, 768, 1024, 8, 8, 3)
    args = (dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8)
    y1 = host(ot.qlinear(*args))
    y2 = host(ot.qlinear(*args))
    assert y1.tobytes() == y2.tobytes()


# --------------------------------------------------------------------------
# End to end on the OPT-125m-shaped workload
# --------------------------------------------------------------------------
@pytest.mark.parametrize("a_bits,w_bits", [(8, 8), (6, 6)])
def test_pipeline_opt125m(a_bits, w_bits):
    wl = synth.WORKLOADS["opt125m_w8a8"]
    batches = list(synth.calibration_batches(wl, 0))
    X = synth.activations(wl, 0, wl.M)
    W = synth.weight(wl, 0)
    b = synth.bias(wl, 0)
    case(f"pipeline opt125m W{w_bits}A{a_bits}")
    ref = O.pipeline(X, W, b, batches, a_bits, w_bits)
    _, z, s, inv_s = ot.calibrate(batches, a_bits)
    Wq, sW, bp = ot.fold_weights(dev(W), dev(b), w_bits, z, s)
    Xq = ot.quantize_act(dev(X), a_bits, z, inv_s)
    Y, acc = ot.qlinear(Xq, Wq, sW, bp, a_bits, w_bits, want_acc=True)
    assert np.array_equal(host(Xq), ref["Xq"])
    assert np.array_equal(host(Wq), ref["Wq"])
    assert np.array_equal(host(acc), ref["acc"])
    assert_fp16_close(host(Y), ref["Y"])


# --------------------------------------------------------------------------
# Prefill tile shapes and the LDS-staged epilogue (Y only, no acc_out): the
# library runs 256 x 256, 320 (channels) x 256 (tokens), 256 x 128 or
# 192 x 256 tiles, whichever its cost model prices lowest.  On a 256-CU
# MI355X the shapes below take, in order, the 320 x 256 tile (256 tiles
# against 320 of 256 x 256), the 256 x 128 tile (less than one pass either
# way), the 192 x 256 tile (one pass, 216 tiles) and the 256 x 256 tile
# (two passes: 205 x 2, against three of 192 x 256); all have ragged M, N
# and K.  The last two repeat the 320 x 256 and 256 x 256 cases with whole
# 16-byte output rows (N a multiple of 8), where the tiles inside M x N take
# the epilogue without per-lane bounds checks and the edge tiles the checked
# one.
# --------------------------------------------------------------------------
PREFILL_TILE_SHAPES = [(500, 40860, 272), (300, 1000, 1040), (2000, 5000, 272), (1025, 9831, 272),
                       (500, 40864, 272), (1025, 9832, 272)]
PREFILL_TILE_ON_256_CUS = {(500, 40860, 272): "prefill 320x256", (300, 1000, 1040): "prefill 256x128",
                           (2000, 5000, 272): "prefill 192x256",
                           (1025, 9831, 272): "prefill 256x256",
                           (500, 40864, 272): "prefill 320x256",
                           (1025, 9832, 272): "prefill 256x256"}


def test_prefill_tiles_all_covered():
    """The tile shapes above are the ones the library runs (on a 256-CU
    MI355X), so each of the three tiles stays covered."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    if cus != 256:
        pytest.skip(f"tile choice depends on the CU count ({cus} here, 256 on MI355X)")
    for shape, name in PREFILL_TILE_ON_256_CUS.items():
        assert ot.ot_qlinear_plan(*shape) == name, shape


@pytest.mark.parametrize("M,N,K", PREFILL_TILE_SHAPES)
@pytest.mark.parametrize("flavour", ["channel", "token", "asym"])
def test_prefill_tiles_staged_epilogue(M, N, K, flavour):
    Xq, Wq, sW, bp = _random_qlinear_inputs(M, N, K, 8, 8, M + 3 * N + 7 * K)
    r = np.random.default_rng(N)
    case(f"prefill staged epilogue {flavour} M={M} N={N} K={K} "
         f"cus={torch.cuda.get_device_properties(0).multi_processor_count} "
         f"plan={ot.ot_qlinear_plan(M, N, K)}")
    if flavour == "channel":
        Y = ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8)
        ref = O.epilogue(O.int_gemm(Xq, Wq), sW, bp)
    elif flavour == "token":
        sX = r.uniform(0.01, 0.2, size=M).astype(np.float32)
        Y = ot.qlinear_per_token(dev(Xq), dev(Wq), dev(sX), dev(sW), dev(bp), 8, 8)
        ref = O.epilogue_per_token(O.int_gemm(Xq, Wq), sX, sW, bp)
    else:
        zW = r.integers(-128, 128, size=N).astype(np.int32)
        Y = ot.qlinear_asym(dev(Xq), dev(Wq), dev(sW), dev(zW), dev(bp), 8, 8)
        ref = O.epilogue(O.int_gemm_asym(Xq, Wq, zW), sW, bp)
    assert_fp16_close(host(Y), ref)


# Every prefill tile at one and two K tiles (K = 48, 128, 144): the next
# tiles' operand loads, spread over the MFMAs of the last K step and the
# following tile's first ones, then all fall past the end of K (zeros into
# a stage nobody reads), and the checkerboard's odd tiles wrap round at once.
PREFILL_SHORT_K = [(500, 40864), (2000, 5000), (1025, 9832), (300, 1000)]


@pytest.mark.parametrize("M,N", PREFILL_SHORT_K)
@pytest.mark.parametrize("K", [48, 128, 144])
def test_prefill_tiles_short_k(M, N, K):
    Xq, Wq, sW, bp = _random_qlinear_inputs(M, N, K, 8, 8, 5 * M + N + K)
    case(f"prefill short K M={M} N={N} K={K} plan={ot.ot_qlinear_plan(M, N, K)}")
    Y, acc = ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8, want_acc=True)
    ref_acc = O.int_gemm(Xq, Wq)
    assert np.array_equal(host(acc), ref_acc)
    Y2 = ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8)  # the staged epilogue
    ref = O.epilogue(ref_acc, sW, bp)
    assert_fp16_close(host(Y), ref)
    assert_fp16_close(host(Y2), ref)


# --------------------------------------------------------------------------
# Split-K decode: 17-64 tokens with at most 32 output channels per CU, given a
# workspace, split K over more workgroups and add their int32 partial sums in
# a second kernel.  The workspace is filled with garbage first (its contents
# need no initialization); outputs must match the oracle and, bit for bit,
# the call without a workspace.
# --------------------------------------------------------------------------
# Split-K plans on 256 CUs (tile height x K runs): 17-32 tokens 32 x 3,
# 64 x 2 (OPT-30B fc2), 96 x 2; 33-64 tokens 32 x 4, 64 x 6, 96 x 3 (OPT-30B
# fc2), 128 x 3 (128-byte K stages)
SPLIT_SHAPES = [(17, 2048, 8192), (32, 7168, 28672), (17, 9216, 16384), (33, 300, 4112),
                (40, 2048, 9216), (64, 7168, 28672), (63, 8192, 9216)]


@pytest.mark.parametrize("M,N,K", SPLIT_SHAPES)
@pytest.mark.parametrize("flavour", ["channel", "token", "asym"])
def test_decode_split_k(M, N, K, flavour):
    nbytes = ot.ot_qlinear_workspace_size(M, N, K)
    case(f"decode split-K {flavour} M={M} N={N} K={K} workspace={nbytes}")
    assert nbytes > 0, "these sizes take the split path on a 256-CU MI355X"
    Xq, Wq, sW, bp = _random_qlinear_inputs(M, N, K, 8, 8, 11 * M + N + K)
    r = np.random.default_rng(M * N)
    ws = torch.from_numpy(r.integers(0, 256, size=nbytes, dtype=np.uint8)).cuda()
    args = [dev(Xq), dev(Wq)]
    if flavour == "channel":
        call = lambda w: ot.qlinear(*args, dev(sW), dev(bp), 8, 8, want_acc=True, workspace=w)
        racc = O.int_gemm(Xq, Wq)
        ref = O.epilogue(racc, sW, bp)
    elif flavour == "token":
        sX = r.uniform(0.01, 0.2, size=M).astype(np.float32)
        call = lambda w: ot.qlinear_per_token(*args, dev(sX), dev(sW), dev(bp), 8, 8,
                                              want_acc=True, workspace=w)
        racc = O.int_gemm(Xq, Wq)
        ref = O.epilogue_per_token(racc, sX, sW, bp)
    else:
        zW = r.integers(-128, 128, size=N).astype(np.int32)
        call = lambda w: ot.qlinear_asym(*args, dev(sW), dev(zW), dev(bp), 8, 8, want_acc=True,
                                         workspace=w)
        racc = O.int_gemm_asym(Xq, Wq, zW)
        ref = O.epilogue(racc, sW, bp)
    Y, acc = call(ws)
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), ref)
    Y0, acc0 = call(None)  # the single-kernel path
    assert torch.equal(Y, Y0) and torch.equal(acc, acc0)
    Y1 = call(ws)[0]  # again, on the previous call's leftovers
    assert torch.equal(Y, Y1)


def test_workspace_too_small_is_rejected_by_the_binding():
    M, N, K = 32, 7168, 28672
    Xq, Wq, sW, bp = (dev(a) for a in _random_qlinear_inputs(M, N, K, 8, 8, 5))
    small = torch.empty(ot.ot_qlinear_workspace_size(M, N, K) - 16, dtype=torch.uint8,
                        device="cuda")
    case("workspace too small")
    with pytest.raises(ValueError):
        ot.qlinear(Xq, Wq, sW, bp, 8, 8, workspace=small)


# --------------------------------------------------------------------------
# HIP graph replay: a prefill call, a decode call and a split-K decode call
# (workspace) captured in one graph, replayed several times with eager work
# and synchronizations in between; every replay must reproduce the eager
# outputs bit for bit (the kernels clear nothing with memset nodes and keep
# no state between calls).
# --------------------------------------------------------------------------
def test_graph_replay_matches_eager():
    shapes = [(300, 772, 1040), (8, 7168, 2064), (40, 2048, 4112)]
    calls = []
    for i, (M, N, K) in enumerate(shapes):
        Xq, Wq, sW, bp = (dev(a) for a in _random_qlinear_inputs(M, N, K, 8, 8, 100 + i))
        Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
        calls.append((Xq, Wq, sW, bp, Y, ot.workspace_for(M, N, K)))
    assert calls[2][5] is not None, "the last shape takes the split-K path"
    # the split-K decode once more on packed weights (registers streamed
    # from the packed layout), into its own output and workspace
    Xq, Wq, sW, bp = calls[2][:4]
    Wp = ot.pack_weights(Wq)
    M, N, K = Xq.shape[0], Wq.shape[0], Wq.shape[1]
    packed = (Xq, Wp, N, sW, bp, torch.empty((M, N), dtype=torch.float16, device="cuda"),
              ot.workspace_for(M, N, K))
    case("graph replay of prefill, decode, split-K decode and packed split-K decode")

    def run():
        for Xq, Wq, sW, bp, Y, ws in calls:
            ot.ot_qlinear(Xq, Wq, sW, bp, 8, 8, Y, workspace=ws)
        Xq, Wp, N, sW, bp, Y, ws = packed
        ot.ot_qlinear_packed(Xq, Wp, N, sW, bp, 8, 8, Y, workspace=ws)
    run()
    torch.cuda.synchronize()
    assert torch.equal(packed[5], calls[2][4])
    outs = [c[4] for c in calls] + [packed[5]]
    ref = [y.clone() for y in outs]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            run()
    torch.cuda.current_stream().wait_stream(s)
    other = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        for y in outs:
            y.zero_()
        other.mul_(1.0001)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for y, r in zip(outs, ref):
            assert torch.equal(y, r), f"replay {rep} differs from the eager outputs"


# --------------------------------------------------------------------------
# Packed decode weights: the layout matches its definition (a re-layout of
# the codes, zero-padded), and ot_qlinear_packed gives ot_qlinear's outputs
# bit for bit on every decode shape, with and without the split-K workspace.
# --------------------------------------------------------------------------
def _pack_reference(Wq):
    N, K = Wq.shape
    G, KS = -(-N // 16), -(-K // 64)
    padded = np.zeros((G * 16, KS * 64), dtype=np.int8)
    padded[:N, :K] = Wq
    # [g][r][s][c][b] -> [g][s][c][r][b]: lane = r + 16 c
    t = padded.reshape(G, 16, KS, 4, 16).transpose(0, 2, 3, 1, 4)
    return t.reshape(-1)


@pytest.mark.parametrize("N,K", [(16, 64), (17, 80), (300, 1040), (7168, 2064)])
def test_pack_weights_layout(N, K):
    Wq = np.random.default_rng(N + K).integers(-128, 128, size=(N, K)).astype(np.int8)
    case(f"pack weights N={N} K={K}")
    Wp = host(ot.pack_weights(dev(Wq)))
    assert np.array_equal(Wp, _pack_reference(Wq))


PACKED_SHAPES = [s for s in QL_SHAPES if s[0] <= 64]


@pytest.mark.parametrize("M,N,K", PACKED_SHAPES)
def test_qlinear_packed_parity(M, N, K):
    Xq, Wq, sW, bp = _random_qlinear_inputs(M, N, K, 8, 8, 7 * M + N + 3 * K)
    case(f"qlinear packed M={M} N={N} K={K}")
    Wp = ot.pack_weights(dev(Wq))
    Y, acc = ot.qlinear_packed(dev(Xq), Wp, N, dev(sW), dev(bp), 8, 8, want_acc=True)
    racc = O.int_gemm(Xq, Wq)
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), O.epilogue(racc, sW, bp))
    Y0 = ot.qlinear(dev(Xq), dev(Wq), dev(sW), dev(bp), 8, 8)
    assert torch.equal(Y, Y0)


@pytest.mark.parametrize("M,N,K", SPLIT_SHAPES)
def test_qlinear_packed_split_k(M, N, K):
    Xq, Wq, sW, bp = _random_qlinear_inputs(M, N, K, 8, 8, 13 * M + N + K)
    case(f"qlinear packed split-K M={M} N={N} K={K}")
    Wp = ot.pack_weights(dev(Wq))
    Y, acc = ot.qlinear_packed(dev(Xq), Wp, N, dev(sW), dev(bp), 8, 8, want_acc=True,
                               workspace=True)
    racc = O.int_gemm(Xq, Wq)
    assert np.array_equal(host(acc), racc)
    assert_fp16_close(host(Y), O.epilogue(racc, sW, bp))

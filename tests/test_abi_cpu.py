"""Host-side checks of libot that need no GPU: the library loads, exports
every entry point include/ot.h declares, and rejects bad arguments before
any HIP call (so these calls are safe without a device)."""
import ctypes
import os
import subprocess

import pytest

from paper_2406_18832_amd import ot

LIB = ot.LIB_PATH


def test_library_is_built():
    assert os.path.exists(LIB), "run __graft_entry__.build() first"


def test_exports_every_declared_symbol():
    declared = ot.declared_symbols()
    assert {"ot_calibrate", "ot_fold_weights", "ot_quantize_act", "ot_qlinear"} <= set(declared)
    L = ctypes.CDLL(LIB)
    for name in declared:
        assert hasattr(L, name), f"{name} declared in ot.h but not exported"
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True)
    exported = {line.split()[-1] for line in out.stdout.splitlines() if " T ot_" in line}
    assert exported == set(declared)


def test_strerror_and_version():
    assert ot.ot_abi_version() == 1
    assert ot.ot_strerror(0) == "ok"
    for code in range(1, 7):
        assert ot.ot_strerror(code) not in ("ok", "unknown status")
    assert ot.ot_strerror(99) == "unknown status"


def test_workspace_size_rule():
    """Scratch only where the decode launch plan splits K: 17..64 tokens,
    runs x M x (N + 1) int32 for 2..8 runs (256 CUs without a GPU, as on
    MI355X).  On the OPT-30B layers only fc2 splits."""
    ws = ot.ot_qlinear_workspace_size
    for M, N, K in [(16, 7168, 28672), (65, 7168, 28672), (4096, 5120, 20480),
                    (0, 7168, 7168), (64, 0, 7168), (64, 7168, 0),
                    # OPT-30B qkv, out, fc1 at 32 and 64 tokens: one kernel
                    (32, 21504, 7168), (64, 21504, 7168), (32, 7168, 7168), (64, 7168, 7168),
                    (32, 28672, 7168), (64, 28672, 7168)]:
        assert ws(M, N, K) == 0, (M, N, K)
    for M, N, K in [(17, 2048, 8192), (33, 300, 4112), (40, 2048, 9216), (63, 8192, 9216),
                    (17, 9216, 16384)]:
        n = ws(M, N, K)
        unit = M * (N + 1) * 4
        assert n % unit == 0 and 2 <= n // unit <= 8, (M, N, K, n)
    # OPT-30B fc2: 64-row tiles x 2 runs at 32 tokens, 96-row x 3 at 64
    assert ws(32, 7168, 28672) == 2 * 32 * 7169 * 4
    assert ws(64, 7168, 28672) == 3 * 64 * 7169 * 4


def test_workspace_size_properties_over_random_shapes():
    """Every split the launch plan picks (17..64 tokens, 256 CUs without a
    GPU): 2..8 runs of at least 1 KiB of K each, on a grid that fits one
    pass over the CUs for some tile height (32..128 rows); never a split
    outside 17..64 tokens."""
    import numpy as np
    r = np.random.default_rng(7)
    ws = ot.ot_qlinear_workspace_size
    for _ in range(400):
        M = int(r.integers(1, 129))
        N = int(r.integers(1, 40000))
        K = int(r.integers(1, 3000)) * 16
        n = ws(M, N, K)
        if not 17 <= M <= 64:
            assert n == 0, (M, N, K)
            continue
        if n == 0:
            continue
        unit = M * (N + 1) * 4
        assert n % unit == 0, (M, N, K, n)
        runs = n // unit
        assert 2 <= runs <= 8, (M, N, K, runs)
        assert (K + 255) // 256 >= 4 * runs, (M, N, K, runs)
        assert any(-(-N // rows) * runs <= 256 for rows in (32, 64, 96, 128)), (M, N, K, runs)


NULL = None


def _qlinear(M, N, K, a_bits=8, w_bits=8):
    return ot.lib().ot_qlinear(NULL, NULL, NULL, NULL, M, N, K, a_bits, w_bits, NULL, NULL,
                               NULL, NULL)


@pytest.mark.parametrize("args,code", [
    ((4, 8, 32, 9, 8), ot.OT_EINVAL),      # a_bits out of range
    ((4, 8, 32, 8, 1), ot.OT_EINVAL),      # w_bits out of range
    ((-1, 8, 32, 8, 8), ot.OT_EINVAL),     # negative M
    ((4, 8, 24, 8, 8), ot.OT_ESHAPE),      # K not a multiple of 16
    ((4, 8, 0, 8, 8), ot.OT_ESHAPE),       # K = 0
    ((4, 0, 32, 8, 8), ot.OT_ESHAPE),      # N = 0
    ((4, 8, 133152, 8, 8), ot.OT_ERANGE),  # K * 127 * 127 >= 2^31
    ((4, 8, 2234640, 6, 6), ot.OT_ERANGE),  # K * 31 * 31 >= 2^31
    ((1 << 30, 1 << 21, 32, 8, 8), ot.OT_ESHAPE),  # more prefill tiles than a 32-bit grid
    ((0, 8, 32, 8, 8), ot.OT_OK),          # M = 0 is a no-op
    ((4, 8, 32, 8, 8), ot.OT_EINVAL),      # null pointers with work to do
])
def test_qlinear_argument_checks(args, code):
    assert _qlinear(*args) == code


def test_qlinear_w6a6_range_accepts_large_k():
    # the same K that overflows at W8A8 is fine at W6A6, up to the null check
    assert _qlinear(4, 8, 133152, 6, 6) == ot.OT_EINVAL


def test_quantize_act_argument_checks():
    L = ot.lib()
    assert L.ot_quantize_act(NULL, 4, 24, 8, NULL, NULL, NULL, NULL) == ot.OT_ESHAPE
    assert L.ot_quantize_act(NULL, 4, 32, 1, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert L.ot_quantize_act(NULL, 0, 32, 8, NULL, NULL, NULL, NULL) == ot.OT_OK
    assert L.ot_quantize_act(NULL, 4, 32, 8, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    # misaligned (but non-null) pointers are rejected before any launch
    assert L.ot_quantize_act(1, 4, 32, 8, 16, 16, 16, NULL) == ot.OT_EINVAL


def test_ln_quantize_act_argument_checks():
    L = ot.lib()
    f = L.ot_ln_quantize_act
    nan = float("nan")
    assert f(NULL, 4, 24, NULL, NULL, 1e-5, 8, NULL, NULL, NULL, NULL) == ot.OT_ESHAPE
    assert f(NULL, 4, 65536 + 16, NULL, NULL, 1e-5, 8, NULL, NULL, NULL, NULL) == ot.OT_ESHAPE
    assert f(NULL, 4, 32, NULL, NULL, 1e-5, 9, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(NULL, 4, 32, NULL, NULL, -1e-5, 8, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(NULL, 4, 32, NULL, NULL, nan, 8, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(NULL, 4, 32, NULL, NULL, float("inf"), 8, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(NULL, 0, 32, NULL, NULL, 1e-5, 8, NULL, NULL, NULL, NULL) == ot.OT_OK
    assert f(NULL, 4, 32, NULL, NULL, 1e-5, 8, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(16, 4, 32, 16, 16, 1e-5, 8, 16, 16, 8, NULL) == ot.OT_EINVAL  # misaligned Xq


def test_per_token_argument_checks():
    L = ot.lib()
    q = L.ot_quantize_act_per_token
    assert q(NULL, 4, 24, 8, NULL, NULL, NULL) == ot.OT_ESHAPE
    assert q(NULL, 4, 65536 + 16, 8, NULL, NULL, NULL) == ot.OT_ESHAPE
    assert q(NULL, 4, 32, 1, NULL, NULL, NULL) == ot.OT_EINVAL
    assert q(NULL, 0, 32, 8, NULL, NULL, NULL) == ot.OT_OK
    assert q(NULL, 4, 32, 8, NULL, NULL, NULL) == ot.OT_EINVAL
    assert q(16, 4, 32, 8, 16, 8, NULL) == ot.OT_EINVAL  # misaligned sX
    f = L.ot_fold_weights_per_token
    assert f(NULL, NULL, NULL, 8, 32, 8, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(16, NULL, NULL, 0, 32, 8, 16, 16, 16, NULL) == ot.OT_ESHAPE
    assert f(16, NULL, NULL, 8, 32, 9, 16, 16, 16, NULL) == ot.OT_EINVAL
    g = L.ot_qlinear_per_token
    assert g(NULL, NULL, NULL, NULL, NULL, 4, 8, 24, 8, 8, NULL, NULL, NULL, NULL) == ot.OT_ESHAPE
    assert g(NULL, NULL, NULL, NULL, NULL, 4, 8, 133152, 8, 8, NULL, NULL, NULL, NULL) == ot.OT_ERANGE
    assert g(NULL, NULL, NULL, NULL, NULL, 0, 8, 32, 8, 8, NULL, NULL, NULL, NULL) == ot.OT_OK
    assert g(16, 16, NULL, 16, 16, 4, 8, 32, 8, 8, 16, NULL, NULL, NULL) == ot.OT_EINVAL


def test_asym_argument_checks():
    L = ot.lib()
    f = L.ot_fold_weights_asym
    assert f(NULL, NULL, 8, 32, 8, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert f(16, NULL, 0, 32, 8, 16, 16, 16, 16, 16, 16, NULL) == ot.OT_ESHAPE
    assert f(16, NULL, 8, 32, 1, 16, 16, 16, 16, 16, 16, NULL) == ot.OT_EINVAL
    g = L.ot_qlinear_asym
    assert g(NULL, NULL, NULL, NULL, NULL, 4, 8, 24, 8, 8, NULL, NULL, NULL, NULL) == ot.OT_ESHAPE
    # K qa 2^w_bits >= 2^31: 66064 * 127 * 256 > 2^31, 66048 * 127 * 256 < 2^31
    assert g(NULL, NULL, NULL, NULL, NULL, 4, 8, 66064, 8, 8, NULL, NULL, NULL, NULL) == ot.OT_ERANGE
    assert g(NULL, NULL, NULL, NULL, NULL, 0, 8, 66048, 8, 8, NULL, NULL, NULL, NULL) == ot.OT_OK
    assert g(16, 16, 16, NULL, 16, 4, 8, 32, 8, 8, 16, NULL, NULL, NULL) == ot.OT_EINVAL


def test_calibrate_and_fold_argument_checks():
    L = ot.lib()
    assert L.ot_calibrate(NULL, 4, 32, 8, 1, NULL, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert L.ot_calibrate(16, 0, 32, 8, 1, 16, 16, 16, 16, NULL) == ot.OT_ESHAPE
    assert L.ot_calibrate(16, 4, 32, 9, 1, 16, 16, 16, 16, NULL) == ot.OT_EINVAL
    assert L.ot_fold_weights(NULL, NULL, 8, 32, 8, NULL, NULL, NULL, NULL, NULL, NULL) == ot.OT_EINVAL
    assert L.ot_fold_weights(16, NULL, 0, 32, 8, 16, 16, 16, 16, 16, NULL) == ot.OT_ESHAPE
    assert L.ot_fold_weights(16, NULL, 8, 32, 0, 16, 16, 16, 16, 16, NULL) == ot.OT_EINVAL


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros((4, 32), dtype=torch.float16)
    with pytest.raises(ValueError):
        ot.ot_quantize_act(x, 8, torch.zeros(32), torch.zeros(32),
                           torch.zeros((4, 32), dtype=torch.int8))


def test_binding_workspace_argument_forms():
    """None/False mean no workspace; a tensor passes through unchanged."""
    import torch
    t = torch.empty(8, dtype=torch.uint8)
    x, w = torch.empty((2, 16), dtype=torch.int8), torch.empty((4, 16), dtype=torch.int8)
    assert ot._ws(None, x, w) is None and ot._ws(False, x, w) is None
    assert ot._ws(t, x, w) is t
    with pytest.raises(ValueError):
        ot._dev_ws(torch.empty(8, dtype=torch.uint8), 2, 4, 16)  # host tensor


def test_packed_weights_size_and_argument_checks():
    sz = ot.ot_packed_weights_size
    assert sz(16, 64) == 1024 and sz(17, 80) == 2 * 2 * 1024 and sz(7168, 7168) == 448 * 112 * 1024
    assert sz(0, 64) == 0 and sz(16, 24) == 0 and sz(16, 0) == 0
    L = ot.lib()
    assert L.ot_pack_weights(None, 16, 24, None, None) == ot.OT_ESHAPE  # K % 16
    assert L.ot_pack_weights(None, 16, 64, None, None) == ot.OT_EINVAL      # null pointers
    q = lambda M, N, K, a=8, w=8: L.ot_qlinear_packed(None, None, None, None, M, N, K, a, w,
                                                       None, None, None, None)
    assert q(65, 8, 32) == ot.OT_ESHAPE      # decode only
    assert q(4, 8, 24) == ot.OT_ESHAPE       # K % 16
    assert q(4, 8, 133152) == ot.OT_ERANGE   # int32 accumulator bound
    assert q(0, 8, 32) == ot.OT_OK           # no work
    assert q(4, 8, 32) == ot.OT_EINVAL       # null pointers
    assert q(4, 8, 32, 9) == ot.OT_EINVAL    # bits


def test_build_info_names_these_sources():
    """The loaded library reports the SHA-256 of the sources and flags it was
    built from; it must be that of the tree under test (a stale build would
    test other code)."""
    info = ot.build_info()
    assert info["arch"] == "gfx950"
    assert len(info["sources_sha256"]) == 64 and int(info["sources_sha256"], 16) >= 0
    assert info["hip"].count(".") == 2
    assert info["matches_sources"], "libot.so was built from other sources: rebuild it"

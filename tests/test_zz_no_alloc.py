"""ot_qlinear_noalloc (the entry point for callers that cannot allocate)
through the C ABI against ot_qlinear with a workspace and against the
oracle: two calls in a row, the second on smaller inputs (so it reads an
array still holding the first call's partial sums), plus the launches that
use no scratch."""
import re

import numpy as np
import pytest
import torch

from oracle import ot_oracle as O
from paper_2406_18832_amd import ot
from tests._tol import assert_fp16_close

pytestmark = pytest.mark.gpu


def _limit():
    with open(ot.HEADER) as f:
        m = re.search(r"#define OT_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", f.read())
    return int(m.group(1)) << int(m.group(2))


def _inputs(M, N, K, seed):
    r = np.random.default_rng(seed)
    Xq = r.integers(-127, 128, size=(M, K)).astype(np.int8)
    Wq = r.integers(-127, 128, size=(N, K)).astype(np.int8)
    sW = (r.uniform(0.5, 2.0, size=N) * 1e-4).astype(np.float32)
    bp = r.normal(0, 1, size=N).astype(np.float32)
    return Xq, Wq, sW, bp


def _check(M, N, K, seed):
    Xq, Wq, sW, bp = _inputs(M, N, K, seed)
    d = [torch.from_numpy(a).cuda() for a in (Xq, Wq, sW, bp)]
    ws = ot.ot_qlinear_workspace_size(M, N, K)
    print(f"[case] noalloc M={M} N={N} K={K} workspace={ws} "
          f"plan={ot.ot_qlinear_plan(M, N, K, with_workspace=True)}", flush=True)
    assert ws <= _limit()
    Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    ot.ot_qlinear_noalloc(d[0], d[1], d[2], d[3], 8, 8, Y, acc)
    Yw, accw = ot.qlinear(*d, 8, 8, want_acc=True, workspace=True)
    torch.cuda.synchronize()
    assert torch.equal(acc, accw) and torch.equal(Y, Yw)
    racc = O.int_gemm(Xq, Wq)
    assert np.array_equal(acc.cpu().numpy(), racc)
    assert_fp16_close(Y.cpu().numpy(), O.epilogue(racc, sW, bp))
    return ws


def test_noalloc_two_split_calls_second_smaller():
    # OPT-30B fc2 at 64 tokens (split K), then a smaller split launch
    assert _check(64, 7168, 28672, 1) > 0
    assert _check(24, 2048, 8192, 2) > 0


def test_noalloc_launches_without_scratch():
    assert _check(8, 3000, 1040, 3) == 0     # decode, no split
    assert _check(300, 1000, 1040, 4) == 0   # prefill


def test_noalloc_largest_split_fits():
    # the largest split a 256-CU device can plan: 64 tokens, 32768 channels
    # over 128-row tiles would take every CU with one run; long K makes the
    # plan split narrower layers instead, up to runs x N = 32768
    worst = max(ot.ot_qlinear_workspace_size(64, n, 65536) for n in (2048, 4096, 8192, 16384))
    assert 0 < worst <= _limit()

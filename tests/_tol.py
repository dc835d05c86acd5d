"""Tolerance helpers shared by the parity tests (no method arithmetic)."""
import numpy as np

# fp16 outputs: within 2 units in the last place of the reference value,
# the unit floored at fp16's smallest subnormal; relative error <= 1e-3.
FP16_ULPS = 2
FP16_MAX_REL = 1e-3


def ulp_fp16(ref):
    a = np.abs(np.asarray(ref, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -24)))
    return np.maximum(np.exp2(e - 10), 2.0 ** -24)


def _within_ulps(got, ref, what):
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    inf_r = ~np.isfinite(r)
    assert np.array_equal(g[inf_r], r[inf_r]), f"{what}: non-finite mismatch"
    fin = ~inf_r
    diff = np.abs(g[fin] - r[fin])
    bound = FP16_ULPS * ulp_fp16(r[fin])
    bad = diff > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {diff.size} outside {FP16_ULPS} ulp; "
                           f"worst diff {diff.max():.3g}")
    rel = diff / np.maximum(np.abs(r[fin]), 2.0 ** -24 * 2 ** 10)
    assert rel.size == 0 or rel.max() <= FP16_MAX_REL, f"{what}: max rel {rel.max():.3g}"
    return int((diff == 0).sum()), int(diff.size)


def assert_fp16_close(got, ref, what="Y", exact=True):
    """The stated bar for fp16 outputs: within FP16_ULPS units in the last
    place of the oracle's value (relative error <= 1e-3).

    With exact=True (every GEMM output here) the outputs must also be the
    oracle's bit patterns: the kernels run the epilogue's float32 steps in
    the oracle's order with contraction off, so any difference, even one
    inside the bar (a fused multiply-add moves Y by at most one unit), is a
    regression.  Returns (matching elements, elements)."""
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert got.dtype == np.float16 and ref.dtype == np.float16, (got.dtype, ref.dtype)
    if np.array_equal(got.view(np.uint16), ref.view(np.uint16)):
        return int(got.size), int(got.size)
    same, total = _within_ulps(got, ref, what)
    same_bits = int((got.view(np.uint16) == ref.view(np.uint16)).sum())
    assert not exact, (f"{what}: within {FP16_ULPS} ulp, but {total - same_bits} of {total} "
                       f"differ from the oracle's bits (epilogue order or contraction changed?)")
    return same, total


def assert_fp32_within_ulps(got, ref, ulps=1, what="bprime"):
    got = np.asarray(got, dtype=np.float32)
    ref = np.asarray(ref, dtype=np.float32)
    gi = got.view(np.int32).astype(np.int64)
    ri = ref.view(np.int32).astype(np.int64)
    # map sign-magnitude bit patterns onto a monotone integer line
    gi = np.where(gi < 0, -(gi & 0x7FFFFFFF), gi)
    ri = np.where(ri < 0, -(ri & 0x7FFFFFFF), ri)
    d = np.abs(gi - ri)
    assert d.max(initial=0) <= ulps, f"{what}: {int((d > ulps).sum())} values beyond {ulps} ulp"
    return int((d == 0).sum()), int(d.size)

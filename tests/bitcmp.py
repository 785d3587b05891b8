"""Bit-pattern comparison of float32 results (tolerance 0 ULP).

+0 and -0 are different results; NaN matches NaN only when the bit patterns are
equal, except where a test asks for ``nan_equal``.
"""
import numpy as np


def _u32(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32).ravel()


def ulp_distance(a, b):
    """Distance in units in the last place along the ordered float32 line."""
    def ordered(u):
        u = u.astype(np.int64)
        return np.where(u & 0x80000000, -(u & 0x7FFFFFFF), u)
    ua, ub = _u32(a), _u32(b)
    return np.abs(ordered(ua) - ordered(ub))


def mismatches(got, want, nan_equal=True):
    g, w = _u32(got), _u32(want)
    bad = g != w
    if nan_equal:
        both_nan = np.isnan(np.asarray(got, np.float32).ravel()) & np.isnan(
            np.asarray(want, np.float32).ravel())
        bad &= ~both_nan
    return np.flatnonzero(bad)


def assert_bits_equal(got, want, what="", nan_equal=True):
    got = np.asarray(got, np.float32)
    want = np.asarray(want, np.float32)
    assert got.shape == want.shape, f"{what}: shape {got.shape} != {want.shape}"
    bad = mismatches(got, want, nan_equal)
    if bad.size:
        i = bad[0]
        idx = tuple(int(x) for x in np.unravel_index(i, got.shape))
        d = ulp_distance(got.ravel()[bad], want.ravel()[bad])
        raise AssertionError(
            f"{what}: {bad.size} of {got.size} outputs differ; first at {idx}: "
            f"got {got.ravel()[i]!r} (0x{_u32(got)[i]:08x}) want {want.ravel()[i]!r} "
            f"(0x{_u32(want)[i]:08x}); max ulp distance {int(d.max())}")

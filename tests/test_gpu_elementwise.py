"""GPU parity of repops_exp / repops_gelu against the CPU oracle (0 ULP) over
binary32 bit patterns: all 2^32 inputs, a strided sweep, the dense core
range, special values, and every elementwise launch shape."""
import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal
from gpu_util import announce, dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2502_19405_amd import repops
    repops.load()
    return repops


SPECIALS = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, -1.0, 88.72283, 88.7229, -87.3,
                     -103.0, -103.97, -104.0, 1e-45, -1e-45, 1.17549435e-38, 3.4028235e38,
                     -3.4028235e38, 20.0, -20.0, -9.6, -10.07, 0.5, 1e-7], np.float32)


def sweep(stride, offset):
    u = np.arange(offset, 2 ** 32, stride, dtype=np.uint64).astype(np.uint32)
    return u.view(np.float32)


@pytest.mark.parametrize("fn", ["exp", "gelu"])
def test_bit_pattern_sweep(rp, fn):
    """Every 61st bit pattern (70.4M inputs, all signs and exponents)."""
    x = np.concatenate([SPECIALS, sweep(61, 5)])
    want = getattr(oracle, fn)(x)
    announce(fn, "sweep", x.size)
    got = host(getattr(rp, fn)(dev(x)))
    assert_bits_equal(got, want, fn)


@pytest.mark.parametrize("fn", ["exp", "gelu"])
def test_dense_core_range(rp, fn):
    """Every 7th binary32 pattern in the range where results are finite and
    mostly normal: exp on [-104, 89], gelu on [-12, 12]."""
    lo, hi = (-104.0, 89.0) if fn == "exp" else (-12.0, 12.0)
    pos = np.arange(0, np.float32(hi).view(np.uint32) + 1, 7, dtype=np.uint32)
    neg = np.arange(0, np.float32(-lo).view(np.uint32) + 1, 7, dtype=np.uint32) | np.uint32(0x80000000)
    x = np.concatenate([pos, neg]).view(np.float32)
    want = getattr(oracle, fn)(x)
    announce(fn, "dense", x.size)
    got = host(getattr(rp, fn)(dev(x)))
    assert_bits_equal(got, want, fn)


@pytest.mark.parametrize("fn", ["exp", "gelu"])
def test_launch_shapes_and_alignment(rp, fn):
    import torch
    g = np.random.default_rng(3)
    x = g.uniform(-30, 30, 100003).astype(np.float32)
    want = getattr(oracle, fn)(x)
    dx = dev(x)
    launches = [None] + [rp.Launch(rp.LAUNCH_ELEMENTWISE, (t, b)) for t, b in
                         ((64, 0), (256, 7), (1024, 0), (512, 1))]
    for launch in launches:
        announce(fn, "launch", launch)
        assert_bits_equal(host(getattr(rp, fn)(dx, launch=launch)), want, str(launch))
        # misaligned views (scalar path) and in place
        off = getattr(rp, fn)(dx[1:], launch=launch)
        assert_bits_equal(host(off), want[1:], "offset view")
        d = dev(x)
        getattr(rp, fn)(d, launch=launch, out=d)
        assert_bits_equal(host(d), want, "in place")
    assert getattr(rp, fn)(torch.empty(0, device="cuda:0")).numel() == 0


def test_copy_keeps_every_bit(rp):
    """The streaming-ceiling copy returns its input bit for bit (signed zeros,
    infinities, NaN payloads, subnormals) for every launch shape, ragged
    lengths, a misaligned view and in place."""
    import torch
    x = np.concatenate([SPECIALS, sweep(65537, 11),
                        np.array([0x7FC00001, 0xFFBADBAD, 0x7F800001, 0x00000001],
                                 np.uint32).view(np.float32)])
    dx = dev(x)
    launches = [None] + [rp.Launch(rp.LAUNCH_ELEMENTWISE, (t, b)) for t, b in
                         ((64, 0), (256, 7), (1024, 0), (512, 1))]
    for launch in launches:
        announce("copy", launch)
        for n in (1, 3, 4, 5, x.size):
            assert_bits_equal(host(rp.copy(dx[:n], launch=launch)), x[:n], f"{launch} n={n}",
                              nan_equal=False)
        assert_bits_equal(host(rp.copy(dx[1:], launch=launch)), x[1:], "offset view",
                          nan_equal=False)
        d = dev(x)
        rp.copy(d, launch=launch, out=d)
        assert_bits_equal(host(d), x, "in place", nan_equal=False)
    assert rp.copy(torch.empty(0, device="cuda:0")).numel() == 0


@pytest.mark.parametrize("fn", ["exp", "gelu"])
def test_exhaustive_all_bit_patterns(rp, fn):
    """Every one of the 2^32 binary32 inputs, in 16 chunks of 2^28: the GPU
    equals the oracle bit for bit (NaN inputs: NaN outputs)."""
    import torch
    chunk = 1 << 28
    ref = getattr(oracle, fn)
    for c in range(16):
        announce(fn, "exhaustive chunk", c)
        base = c * chunk
        # bit patterns base .. base + chunk - 1 as float32 (int64 -> int32 wraps)
        x = (torch.arange(base, base + chunk, dtype=torch.int64, device="cuda:0")
             .to(torch.int32).view(torch.float32))
        got = host(getattr(rp, fn)(x))
        xs = (np.arange(base, base + chunk, dtype=np.uint64).astype(np.uint32)).view(np.float32)
        want = ref(xs)
        assert_bits_equal(got, want, f"{fn} chunk {c}")
        del x, got, xs, want

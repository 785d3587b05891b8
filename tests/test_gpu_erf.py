"""GPU parity of erf and the erf-form GELU (forward and backward) against the
CPU oracle: every one of the 2^32 binary32 inputs, every launch
configuration, misaligned and in-place calls."""
import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal
from gpu_util import announce, dev, host
from paper_2502_19405_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2502_19405_amd import repops
    repops.load()
    return repops


def ew_launches(rp):
    return [("auto", None), ("t64", rp.Launch(rp.LAUNCH_ELEMENTWISE, (64, 0))),
            ("t1024", rp.Launch(rp.LAUNCH_ELEMENTWISE, (1024, 0))),
            ("t256b7", rp.Launch(rp.LAUNCH_ELEMENTWISE, (256, 7)))]


@pytest.mark.parametrize("n", [1, 5, 1000, 1001, 4096 * 3072 + 3])
def test_erf_gelu_erf_all_launches(rp, n):
    g = inputs.rng(1000 + n % 997)
    x = np.concatenate([inputs.normal(g, (n // 2 + 1,), var=9.0),
                        inputs.uniform(g, (n - n // 2 - 1,), -16, 16)])
    dy = inputs.normal(g, (n,), var=1e-2)
    we, wg, wb = oracle.erf(x), oracle.gelu_erf(x), oracle.gelu_erf_backward(x, dy)
    xd, dyd = dev(x), dev(dy)
    for name, launch in ew_launches(rp):
        announce("erf family", n, name)
        assert_bits_equal(host(rp.erf(xd, launch=launch)), we, f"erf {name}")
        assert_bits_equal(host(rp.gelu_erf(xd, launch=launch)), wg, f"gelu_erf {name}")
        assert_bits_equal(host(rp.gelu_erf_backward(xd, dyd, launch=launch)), wb, f"bwd {name}")
    if n > 4:
        announce("erf family misaligned", n)
        pad = lambda a: dev(np.concatenate([np.zeros(1, np.float32), a]))[1:]  # noqa: E731
        assert_bits_equal(host(rp.gelu_erf(pad(x))), wg, "misaligned gelu_erf")
        assert_bits_equal(host(rp.gelu_erf_backward(pad(x), pad(dy))), wb, "misaligned bwd")


def test_erf_family_in_place_and_specials(rp):
    x = np.array([0.0, -0.0, 0.5, -0.5, 0.49999997, 2.5, -2.5, 2.4999998, 10.5, -10.5, 14.9,
                  -14.9, 20.0, -20.0, 1e-30, -1e-30, 1e-45, np.inf, -np.inf, np.nan,
                  3.4e38, -3.4e38], np.float32)
    for fn, ref in (("erf", oracle.erf), ("gelu_erf", oracle.gelu_erf)):
        announce("in place", fn)
        d = dev(x)
        getattr(rp, fn)(d, out=d)
        assert_bits_equal(host(d), ref(x), fn)
    dy = np.full_like(x, 0.75)
    announce("in place gelu_erf_backward")
    d = dev(dy)
    rp.gelu_erf_backward(dev(x), d, out=d)
    assert_bits_equal(host(d), oracle.gelu_erf_backward(x, dy), "bwd over dy")


@pytest.mark.parametrize("fn", ["erf", "gelu_erf", "gelu_erf_grad"])
def test_exhaustive_all_bit_patterns(rp, fn):
    """All 2^32 inputs in 16 chunks of 2^28 (the derivative through the
    backward with dy = 1, where RN(1 * g) = g)."""
    import torch
    chunk = 1 << 28
    for c in range(16):
        announce(fn, "exhaustive chunk", c)
        base = c * chunk
        x = (torch.arange(base, base + chunk, dtype=torch.int64, device="cuda:0")
             .to(torch.int32).view(torch.float32))
        xs = (np.arange(base, base + chunk, dtype=np.uint64).astype(np.uint32)).view(np.float32)
        if fn == "gelu_erf_grad":
            ones = torch.ones_like(x)
            got = host(rp.gelu_erf_backward(x, ones))
            want = oracle.gelu_erf_backward(xs, np.ones_like(xs))
            del ones
        else:
            got = host(getattr(rp, fn)(x))
            want = getattr(oracle, fn)(xs)
        assert_bits_equal(got, want, f"{fn} chunk {c}")
        del x, xs, got, want

"""GPU parity of repops_softmax_rows / repops_layernorm_rows against the CPU
oracle (0 ULP): ragged rows, causal masks, in-place calls, padded leading
dimensions, every row order descriptor, every launch configuration."""
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


def row_launches(rp, W=64, combine=0, cols=0):
    out = [("generic", rp.Launch(rp.LAUNCH_ROWS_GENERIC)), ("auto", None)]
    if W == 64 and combine == 0 and cols <= 4096:
        out += [(f"wave{w}", rp.Launch(rp.LAUNCH_ROWS_WAVE, (w,))) for w in (1, 2, 4, 8)]
    if W == 64 and combine == 0:
        # one row per workgroup, split over S waves (at most 32 values per lane)
        out += [(f"split{S}", rp.Launch(rp.LAUNCH_ROWS_WAVE, (1, S)))
                for S in (2, 4, 8) if cols <= S * 64 * 32]
    return out


COLS = [1, 2, 63, 64, 65, 100, 256, 768, 1000, 1024, 2048, 2049, 3000, 4096, 5000, 8192, 20000]


@pytest.mark.parametrize("cols", COLS)
@pytest.mark.parametrize("period", [0, 7, 37])
def test_softmax_ragged_all_launches(rp, cols, period):
    g = inputs.rng(cols * 10 + period)
    X = inputs.normal(g, (75, cols), var=4.0)
    want = oracle.softmax_rows(X, causal_period=period)
    dX = dev(X)
    for name, launch in row_launches(rp, cols=cols):
        announce("softmax", cols, period, name)
        got = host(rp.softmax_rows(dX, causal_period=period, launch=launch))
        assert_bits_equal(got, want, f"{name} cols={cols} period={period}")


@pytest.mark.parametrize("W,combine", [(1, 0), (16, 0), (128, 0), (1024, 0), (64, 1), (8, 1),
                                       (256, 1)])
def test_softmax_other_orders(rp, W, combine):
    g = inputs.rng(W + combine)
    X = inputs.normal(g, (40, 777), var=4.0)
    for period in (0, 100):
        want = oracle.softmax_rows(X, causal_period=period, row_width=W, row_combine=combine)
        announce("softmax order", W, combine, period)
        got = host(rp.softmax_rows(dev(X), causal_period=period,
                                   order=rp.Order(row_width=W, row_combine=combine)))
        assert_bits_equal(got, want, f"W={W} combine={combine}")


def test_softmax_in_place_and_padded(rp):
    import torch
    g = inputs.rng(5)
    X = inputs.normal(g, (33, 300), var=4.0)
    want = oracle.softmax_rows(X, causal_period=50)
    for name, launch in row_launches(rp, cols=300):
        announce("softmax in place", name)
        d = dev(X)
        rp.softmax_rows(d, causal_period=50, launch=launch, out=d)
        assert_bits_equal(host(d), want, name)
        big = torch.full((33, 320), float("nan"), device="cuda:0")
        big[:, :300] = dev(X)
        out = torch.full((33, 310), -7.0, device="cuda:0")
        rp.softmax_rows(big[:, :300], causal_period=50, launch=launch, out=out[:, :300])
        o = host(out)
        assert_bits_equal(o[:, :300], want, name + " padded")
        assert (o[:, 300:] == -7.0).all()


def test_softmax_masked_entries_are_never_read(rp):
    """Causal skipping: masked inputs hold NaN and infinities, outputs are the
    same as with finite masked inputs (masked outputs +0)."""
    g = inputs.rng(6)
    X = inputs.normal(g, (64, 64), var=4.0)
    want = oracle.softmax_rows(X, causal_period=64)
    Xp = X.copy()
    iu = np.triu_indices(64, 1)
    Xp[iu] = np.where(np.arange(iu[0].size) % 2, np.nan, np.inf).astype(np.float32)
    for name, launch in row_launches(rp, cols=64):
        announce("softmax masked", name)
        got = host(rp.softmax_rows(dev(Xp), causal_period=64, launch=launch))
        assert_bits_equal(got, want, name)


def test_softmax_closed_forms(rp):
    X = np.full((4, 256), 3.25, np.float32)
    got = host(rp.softmax_rows(dev(X)))
    assert (got == np.float32(1) / np.float32(256)).all()
    Y = np.full((1, 300), -200.0, np.float32)
    Y[0, 0] = 0
    got = host(rp.softmax_rows(dev(Y)))
    assert got[0, 0] == 1 and (got[0, 1:] == 0).all()


@pytest.mark.parametrize("cols", [1, 2, 5, 64, 100, 768, 1024, 2048, 3000, 4096, 8192, 9000])
@pytest.mark.parametrize("affine", ["both", "gamma", "beta", "none"])
def test_layernorm_ragged_all_launches(rp, cols, affine):
    g = inputs.rng(cols + len(affine))
    X = inputs.normal(g, (70, cols))
    X[3] = 1.5  # constant row: d = +0, y = beta
    gamma = (1 + inputs.uniform(g, (cols,), -0.1, 0.1)) if affine in ("both", "gamma") else None
    beta = inputs.uniform(g, (cols,), -0.1, 0.1) if affine in ("both", "beta") else None
    want, mean, rstd = oracle.layernorm_rows(X, gamma, beta, eps=1e-5, with_stats=True)
    import torch
    for name, launch in row_launches(rp, cols=cols):
        announce("layernorm", cols, affine, name)
        m = torch.empty(70, device="cuda:0")
        r = torch.empty(70, device="cuda:0")
        got = rp.layernorm_rows(dev(X), None if gamma is None else dev(gamma),
                                None if beta is None else dev(beta), eps=1e-5, launch=launch,
                                mean_out=m, rstd_out=r)
        assert_bits_equal(host(got), want, f"{name} cols={cols}")
        assert_bits_equal(host(m), mean, "mean")
        assert_bits_equal(host(r), rstd, "rstd")


@pytest.mark.parametrize("W,combine", [(1, 0), (32, 0), (512, 0), (64, 1), (4, 1)])
def test_layernorm_other_orders(rp, W, combine):
    g = inputs.rng(W * 3 + combine)
    X = inputs.normal(g, (30, 900), var=9.0)
    gamma = 1 + inputs.uniform(g, (900,), -0.1, 0.1)
    beta = inputs.uniform(g, (900,), -0.1, 0.1)
    want = oracle.layernorm_rows(X, gamma, beta, row_width=W, row_combine=combine)
    announce("layernorm order", W, combine)
    got = host(rp.layernorm_rows(dev(X), dev(gamma), dev(beta),
                                 order=rp.Order(row_width=W, row_combine=combine)))
    assert_bits_equal(got, want, f"W={W} combine={combine}")


def test_layernorm_sqrt_and_division_coverage(rp):
    """Two-element rows (0, 2b) give mean b, var = RN(b^2) exactly, so with
    eps = 0 the square root and reciprocal run on a million variances spread
    over the whole normal exponent range."""
    g = inputs.rng(9)
    e = g.uniform(-60, 60, 1 << 20)
    b = (np.exp2(e) * g.uniform(1, 2, e.size)).astype(np.float32)
    X = np.stack([np.zeros_like(b), 2 * b], axis=1).astype(np.float32)
    import torch
    for eps in (0.0, 1e-5):
        want, mean, rstd = oracle.layernorm_rows(X, eps=eps, with_stats=True)
        for name, launch in row_launches(rp, cols=2):
            announce("layernorm sqrt coverage", eps, name)
            r = torch.empty(X.shape[0], device="cuda:0")
            got = rp.layernorm_rows(dev(X), eps=eps, launch=launch, rstd_out=r)
            assert_bits_equal(host(r), rstd, f"rstd {name}")
            assert_bits_equal(host(got), want, f"y {name}")


def test_layernorm_in_place(rp):
    g = inputs.rng(10)
    X = inputs.normal(g, (50, 768))
    want = oracle.layernorm_rows(X)
    for name, launch in row_launches(rp, cols=768):
        announce("layernorm in place", name)
        d = dev(X)
        rp.layernorm_rows(d, launch=launch, out=d)
        assert_bits_equal(host(d), want, name)

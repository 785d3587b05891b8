"""GPU parity of the training-step operators against the CPU oracle (0 ULP):
softmax backward, LayerNorm backward (input and parameter gradients), GELU
backward and the Adam / AdamW step -- ragged sizes, causal masks, every row
order, several contraction block lengths, in-place calls, padded leading
dimensions, every launch configuration, and the shapes of the DistilBERT and
Llama training programs."""
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


def ew_launches(rp):
    return [("auto", None), ("t64", rp.Launch(rp.LAUNCH_ELEMENTWISE, (64, 0))),
            ("t1024", rp.Launch(rp.LAUNCH_ELEMENTWISE, (1024, 0))),
            ("t256b7", rp.Launch(rp.LAUNCH_ELEMENTWISE, (256, 7)))]


COLS = [1, 2, 63, 64, 65, 100, 256, 768, 1000, 1024, 2048, 2049, 3000, 4096, 4097, 8192, 20000]


# --------------------------------------------------------------------------
# softmax backward
# --------------------------------------------------------------------------

def softmax_pair(seed, rows, cols, period=0):
    g = inputs.rng(seed)
    X = inputs.normal(g, (rows, cols), var=4.0)
    Y = oracle.softmax_rows(X, causal_period=period)
    dY = inputs.normal(g, (rows, cols))
    return Y, dY


@pytest.mark.parametrize("cols", COLS)
@pytest.mark.parametrize("period", [0, 7, 37])
def test_softmax_backward_ragged_all_launches(rp, cols, period):
    Y, dY = softmax_pair(cols * 10 + period, 75, cols, period)
    want = oracle.softmax_backward_rows(Y, dY, causal_period=period)
    dYd, Yd = dev(dY), dev(Y)
    for name, launch in row_launches(rp, cols=cols):
        announce("softmax_backward", cols, period, name)
        got = host(rp.softmax_backward_rows(Yd, dYd, causal_period=period, launch=launch))
        assert_bits_equal(got, want, f"{name} cols={cols} period={period}")


@pytest.mark.parametrize("W,combine", [(1, 0), (16, 0), (128, 0), (1024, 0), (64, 1), (8, 1),
                                       (256, 1)])
def test_softmax_backward_other_orders(rp, W, combine):
    Y, dY = softmax_pair(300 + W + combine, 40, 777)
    for period in (0, 100):
        want = oracle.softmax_backward_rows(Y, dY, causal_period=period, row_width=W,
                                            row_combine=combine)
        announce("softmax_backward order", W, combine, period)
        got = host(rp.softmax_backward_rows(dev(Y), dev(dY), causal_period=period,
                                            order=rp.Order(row_width=W, row_combine=combine)))
        assert_bits_equal(got, want, f"W={W} combine={combine}")


def test_softmax_backward_in_place_and_padded(rp):
    import torch
    Y, dY = softmax_pair(301, 33, 300, 50)
    want = oracle.softmax_backward_rows(Y, dY, causal_period=50)
    for name, launch in row_launches(rp, cols=300):
        announce("softmax_backward in place", name)
        d = dev(dY)
        rp.softmax_backward_rows(dev(Y), d, causal_period=50, launch=launch, out=d)
        assert_bits_equal(host(d), want, name + " dX = dY")
        y = dev(Y)
        rp.softmax_backward_rows(y, dev(dY), causal_period=50, launch=launch, out=y)
        assert_bits_equal(host(y), want, name + " dX = Y")
        big = torch.full((33, 320), float("nan"), device="cuda:0")
        big[:, :300] = dev(Y)
        bigd = torch.full((33, 340), float("nan"), device="cuda:0")
        bigd[:, :300] = dev(dY)
        out = torch.full((33, 310), -7.0, device="cuda:0")
        rp.softmax_backward_rows(big[:, :300], bigd[:, :300], causal_period=50, launch=launch,
                                 out=out[:, :300])
        o = host(out)
        assert_bits_equal(o[:, :300], want, name + " padded")
        assert (o[:, 300:] == -7.0).all()


def test_softmax_backward_masked_entries_are_never_read(rp):
    Y, dY = softmax_pair(302, 64, 256, 64)
    want = oracle.softmax_backward_rows(Y, dY, causal_period=64)
    Yp, dYp = Y.copy(), dY.copy()
    mask = np.arange(256)[None, :] > (np.arange(64) % 64)[:, None]
    Yp[mask] = np.nan
    dYp[mask] = np.inf
    for name, launch in row_launches(rp, cols=256):
        announce("softmax_backward masked reads", name)
        got = host(rp.softmax_backward_rows(dev(Yp), dev(dYp), causal_period=64, launch=launch))
        assert_bits_equal(got, want, name)


def test_softmax_backward_llama_attention_shape(rp):
    """Causal attention probabilities of the Llama program: 4 x 32 heads x
    1024 queries, 1024 keys (131072 rows), every row compared."""
    rows, cols = 4 * 32 * 1024, 1024
    g = inputs.rng(303)
    X = inputs.normal(g, (rows, cols), var=1.0)
    Y = oracle.softmax_rows(X, causal_period=1024)
    del X
    dY = inputs.normal(g, (rows, cols), var=1e-4)
    want = oracle.softmax_backward_rows(Y, dY, causal_period=1024)
    announce("softmax_backward llama", rows, cols)
    got = host(rp.softmax_backward_rows(dev(Y), dev(dY), causal_period=1024))
    assert_bits_equal(got, want, "llama attention softmax backward")


# --------------------------------------------------------------------------
# LayerNorm backward
# --------------------------------------------------------------------------

def ln_case(seed, rows, cols, with_gamma=True):
    g = inputs.rng(seed)
    X = inputs.normal(g, (rows, cols), var=2.0) + np.float32(0.5)
    gamma = (inputs.normal(g, (cols,), var=0.1) + np.float32(1.0)) if with_gamma else None
    beta = inputs.normal(g, (cols,), var=0.1) if with_gamma else None
    _, mean, rstd = oracle.layernorm_rows(X, gamma, beta, with_stats=True)
    dY = inputs.normal(g, (rows, cols), var=1e-2)
    return X, dY, mean, rstd, gamma


def run_lnb(rp, X, dY, mean, rstd, gamma, order=None, launch=None, workspace=None):
    r = rp.layernorm_backward_rows(dev(X), dev(dY), dev(mean), dev(rstd),
                                   None if gamma is None else dev(gamma), order=order,
                                   launch=launch, workspace=workspace)
    return tuple(host(t) for t in r)


@pytest.mark.parametrize("cols", COLS)
def test_layernorm_backward_ragged_all_launches(rp, cols):
    for rows, with_gamma in ((75, True), (130, False)):
        X, dY, mean, rstd, gamma = ln_case(cols * 3 + rows, rows, cols, with_gamma)
        want = oracle.layernorm_backward_rows(X, dY, mean, rstd, gamma)
        for name, launch in row_launches(rp, cols=cols):
            announce("layernorm_backward", rows, cols, with_gamma, name)
            got = run_lnb(rp, X, dY, mean, rstd, gamma, launch=launch)
            for a, b, what in zip(got, want, ("dX", "dgamma", "dbeta")):
                assert_bits_equal(a, b, f"{name} {what} rows={rows} cols={cols}")


@pytest.mark.parametrize("W,combine,k_block", [(1, 0, 64), (16, 0, 0), (1024, 0, 16),
                                               (64, 1, 128), (8, 1, 1), (256, 1, 64),
                                               (64, 0, 0), (64, 0, 7)])
def test_layernorm_backward_other_orders(rp, W, combine, k_block):
    X, dY, mean, rstd, gamma = ln_case(400 + W + combine + k_block, 150, 777)
    want = oracle.layernorm_backward_rows(X, dY, mean, rstd, gamma, row_width=W,
                                          row_combine=combine, k_block=k_block)
    announce("layernorm_backward order", W, combine, k_block)
    got = run_lnb(rp, X, dY, mean, rstd, gamma,
                  order=rp.Order(row_width=W, row_combine=combine, k_block=k_block))
    for a, b, what in zip(got, want, ("dX", "dgamma", "dbeta")):
        assert_bits_equal(a, b, f"W={W} combine={combine} k_block={k_block} {what}")


def test_layernorm_backward_in_place_workspace_and_partial_requests(rp):
    import torch
    X, dY, mean, rstd, gamma = ln_case(401, 200, 300)
    want = oracle.layernorm_backward_rows(X, dY, mean, rstd, gamma)
    need = rp.layernorm_backward_workspace(200, 300)
    assert need == 2 * 4 * 300 * 4
    ws = torch.full((need // 4 + 5,), float("nan"), device="cuda:0")
    for name, launch in row_launches(rp, cols=300):
        announce("layernorm_backward in place", name)
        d = dev(dY)
        dx, dg, db = rp.layernorm_backward_rows(dev(X), d, dev(mean), dev(rstd), dev(gamma),
                                                launch=launch, dx_out=d, workspace=ws)
        assert_bits_equal(host(dx), want[0], name + " dX = dY")
        assert_bits_equal(host(dg), want[1], name + " dgamma")
        assert_bits_equal(host(db), want[2], name + " dbeta")
        x = dev(X)
        dx, _, _ = rp.layernorm_backward_rows(x, dev(dY), dev(mean), dev(rstd), dev(gamma),
                                              launch=launch, dx_out=x, need_params=False)
        assert_bits_equal(host(dx), want[0], name + " dX = X")
    announce("layernorm_backward params only")
    _, dg, db = rp.layernorm_backward_rows(dev(X), dev(dY), dev(mean), dev(rstd), dev(gamma),
                                           need_dx=False)
    assert_bits_equal(host(dg), want[1], "params only dgamma")
    assert_bits_equal(host(db), want[2], "params only dbeta")


@pytest.mark.parametrize("cols", [1500, 2048, 3000, 4096])
def test_layernorm_backward_in_place_wide_rows(rp, cols):
    """Wide rows in place: the multi-workgroup kernel (other workgroups read
    the rows dX replaces) must not be taken; the parameter gradients come
    first, then dX over X or dY.  LayerNorm and RMSNorm, 3 and 70 row blocks."""
    for rows in (150, 4470):
        X, dY, mean, rstd, gamma = ln_case(cols + rows, rows, cols)
        want = oracle.layernorm_backward_rows(X, dY, mean, rstd, gamma)
        for which in ("dY", "X"):
            announce("layernorm_backward in place wide", rows, cols, which)
            x, d = dev(X), dev(dY)
            dx, dg, db = rp.layernorm_backward_rows(x, d, dev(mean), dev(rstd), dev(gamma),
                                                    dx_out=d if which == "dY" else x)
            assert_bits_equal(host(dx), want[0], f"dX = {which} {rows}x{cols}")
            assert_bits_equal(host(dg), want[1], f"dgamma, dX = {which} {rows}x{cols}")
            assert_bits_equal(host(db), want[2], f"dbeta, dX = {which} {rows}x{cols}")
        _, rstd2 = oracle.rmsnorm_rows(X, gamma, with_stats=True)
        want = oracle.rmsnorm_backward_rows(X, dY, rstd2, gamma)
        announce("rmsnorm_backward in place wide", rows, cols)
        d = dev(dY)
        dx, dg = rp.rmsnorm_backward_rows(dev(X), d, dev(rstd2), dev(gamma), dx_out=d)
        assert_bits_equal(host(dx), want[0], f"rms dX = dY {rows}x{cols}")
        assert_bits_equal(host(dg), want[1], f"rms dgamma, dX = dY {rows}x{cols}")


def test_layernorm_backward_no_rows_gives_zero_parameter_gradients(rp):
    import torch
    announce("layernorm_backward rows=0")
    X = torch.empty((0, 40), device="cuda:0")
    z = torch.empty(0, device="cuda:0")
    _, dg, db = rp.layernorm_backward_rows(X, X, z, z, None, need_dx=False)
    assert (host(dg).view(np.uint32) == 0).all() and (host(db).view(np.uint32) == 0).all()


def test_layernorm_backward_distilbert_shape(rp):
    """The DistilBERT LayerNorm: 4096 tokens x 768, every output compared."""
    X, dY, mean, rstd, gamma = ln_case(402, 4096, 768)
    want = oracle.layernorm_backward_rows(X, dY, mean, rstd, gamma)
    announce("layernorm_backward distilbert")
    got = run_lnb(rp, X, dY, mean, rstd, gamma)
    for a, b, what in zip(got, want, ("dX", "dgamma", "dbeta")):
        assert_bits_equal(a, b, f"distilbert {what}")


# Row-block counts on both sides of 256: with fewer, the automatic launch
# spreads each block's rows and columns over several workgroups (block counts
# with and without a multiple of 8, k_block 1 and k_block past the last row);
# with more, one workgroup per block stages rows in LDS, unless the rows are
# too wide for its stage (over 2048 columns), when the blocks are spread as
# with few.  Rows over 2048 columns take a pair of waves per row.  RMSNorm, and
# an explicit wave launch on the same inputs.
@pytest.mark.parametrize("rows,cols,k_block", [(512, 1024, 64), (1000, 96, 16), (2048, 300, 128),
                                               (130, 1000, 1), (777, 64, 4096), (4096, 17, 64),
                                               (8 * 64, 768, 64), (255 * 16 - 3, 200, 16),
                                               (110 * 64 - 5, 768, 64), (300, 200, 1),
                                               (256 * 16 + 5, 96, 16), (256 * 64, 768, 64),
                                               (4096, 2048, 64), (1000, 3000, 16),
                                               (4096, 4096, 64), (258 * 16 - 5, 2100, 16),
                                               (70, 4096, 4096)])
def test_layernorm_backward_row_block_counts(rp, rows, cols, k_block):
    X, dY, mean, rstd, gamma = ln_case(rows + cols + k_block, rows, cols)
    order = rp.Order(k_block=k_block)
    want = oracle.layernorm_backward_rows(X, dY, mean, rstd, gamma, k_block=k_block)
    for name, launch in (("auto", None), ("wave4", rp.Launch(rp.LAUNCH_ROWS_WAVE, (4,)))):
        announce("layernorm_backward few blocks", rows, cols, k_block, name)
        got = run_lnb(rp, X, dY, mean, rstd, gamma, order=order, launch=launch)
        for a, b, what in zip(got, want, ("dX", "dgamma", "dbeta")):
            assert_bits_equal(a, b, f"{name} {what} {rows}x{cols} k_block={k_block}")
    announce("rmsnorm_backward few blocks", rows, cols, k_block)
    _, rstd2 = oracle.rmsnorm_rows(X, gamma, with_stats=True)
    want = oracle.rmsnorm_backward_rows(X, dY, rstd2, gamma, k_block=k_block)
    dx, dg = rp.rmsnorm_backward_rows(dev(X), dev(dY), dev(rstd2), dev(gamma), order=order)
    assert_bits_equal(host(dx), want[0], f"rms dX {rows}x{cols} k_block={k_block}")
    assert_bits_equal(host(dg), want[1], f"rms dgamma {rows}x{cols} k_block={k_block}")


# --------------------------------------------------------------------------
# bias gradient (column sums)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols,k_block", [(75, 100, 64), (4096, 768, 64), (4096, 3072, 64),
                                               (300, 77, 0), (300, 77, 7), (0, 40, 64),
                                               (64, 5000, 64), (1, 3, 64)])
def test_colsum_rows(rp, rows, cols, k_block):
    import torch
    g = inputs.rng(1050 + rows + k_block)
    X = inputs.normal(g, (rows, cols))
    want = oracle.colsum_rows(X, k_block)
    announce("colsum", rows, cols, k_block)
    got = rp.colsum_rows(dev(X) if rows else torch.empty((0, cols), device="cuda:0"),
                         order=rp.Order(k_block=k_block))
    assert_bits_equal(host(got), want, f"{rows}x{cols} k_block={k_block}")
    if rows:  # the same as the product ones^T X
        ones = torch.ones((1, rows), device="cuda:0")
        via = rp.matmul(ones, dev(X), order=rp.Order(k_block=k_block))
        assert_bits_equal(host(via)[0], want, "ones^T X")


# --------------------------------------------------------------------------
# GELU backward
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 3, 4, 5, 1000, 1001, 4096 * 3072 + 3])
def test_gelu_backward_all_launches(rp, n):
    g = inputs.rng(500 + n % 1000)
    x = inputs.normal(g, (n,), var=9.0)
    dy = inputs.normal(g, (n,), var=1e-2)
    want = oracle.gelu_backward(x, dy)
    xd, dyd = dev(x), dev(dy)
    for name, launch in ew_launches(rp):
        announce("gelu_backward", n, name)
        assert_bits_equal(host(rp.gelu_backward(xd, dyd, launch=launch)), want, f"{name} n={n}")
    if n > 4:  # misaligned views take the scalar path
        announce("gelu_backward misaligned", n)
        got = host(rp.gelu_backward(dev(np.concatenate([np.zeros(1, np.float32), x]))[1:], dyd))
        assert_bits_equal(got, want, "misaligned")


def test_gelu_backward_in_place_and_special_values(rp):
    x = np.array([0.0, -0.0, 1.0, -1.0, 3.0, -3.0, 10.0, -10.0, 44.0, -44.0, 88.0, -88.0,
                  1e-30, -1e-30, 1e-45, np.inf, -np.inf, np.nan, 3.4e38, -3.4e38], np.float32)
    dy = np.ones_like(x) * np.float32(0.75)
    want = oracle.gelu_backward(x, dy)
    for which in ("x", "dy"):
        announce("gelu_backward in place", which)
        xd, dyd = dev(x), dev(dy)
        out = xd if which == "x" else dyd
        rp.gelu_backward(xd, dyd, out=out)
        assert_bits_equal(host(out), want, f"in place over {which}")


def test_gelu_backward_exhaustive_unit_gradient(rp):
    """dy = 1 over all 2^32 binary32 inputs: the GPU derivative equals the
    oracle's bit for bit, in 16 chunks of 2^28."""
    import torch
    chunk = 1 << 28
    for c in range(16):
        announce("gelu_backward exhaustive chunk", c)
        base = c * chunk
        x = (torch.arange(base, base + chunk, dtype=torch.int64, device="cuda:0")
             .to(torch.int32).view(torch.float32))
        ones = torch.ones_like(x)
        got = host(rp.gelu_backward(x, ones))
        xs = (np.arange(base, base + chunk, dtype=np.uint64).astype(np.uint32)).view(np.float32)
        want = oracle.gelu_backward(xs, np.ones_like(xs))
        assert_bits_equal(got, want, f"chunk {c}")
        del x, ones, got, xs, want


# --------------------------------------------------------------------------
# Adam / AdamW
# --------------------------------------------------------------------------

ADAM_CASES = [(0.0, True), (0.01, True), (0.01, False), (0.1, False)]


@pytest.mark.parametrize("wd,decoupled", ADAM_CASES)
@pytest.mark.parametrize("n", [1, 3, 4, 7, 1000, 1001, 65536 + 5])
def test_adam_steps_all_launches(rp, n, wd, decoupled):
    g = inputs.rng(600 + n % 997 + int(wd * 100) + decoupled)
    p0 = inputs.normal(g, (n,), var=0.02 ** 2 * 100)
    grads = [inputs.normal(g, (n,), var=1e-4) for _ in range(4)]
    for name, launch in ew_launches(rp):
        announce("adam", n, wd, decoupled, name)
        p, m, v = p0.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32)
        pd, md, vd = dev(p), dev(m), dev(v)
        for t, gr in enumerate(grads, start=1):
            p, m, v = oracle.adam_step(p, gr, m, v, 1e-3, 0.9, 0.999, 1e-8, wd, t, decoupled)
            rp.adam_step(pd, dev(gr), md, vd, 1e-3, 0.9, 0.999, 1e-8, wd, t, decoupled,
                         launch=launch)
            assert_bits_equal(host(pd), p, f"{name} p step {t}")
            assert_bits_equal(host(md), m, f"{name} m step {t}")
            assert_bits_equal(host(vd), v, f"{name} v step {t}")


@pytest.mark.parametrize("step", [1, 2, 10, 1000, 123457])
def test_adam_late_steps_and_other_hyperparameters(rp, step):
    g = inputs.rng(700 + step % 1000)
    n = 4099
    p = inputs.normal(g, (n,))
    gr = inputs.normal(g, (n,), var=1e-2)
    m = inputs.normal(g, (n,), var=1e-4)
    v = np.abs(inputs.normal(g, (n,), var=1e-6))
    for hp in ((3e-4, 0.9, 0.95, 1e-6, 0.1, True), (1e-2, 0.5, 0.9999, 1e-8, 0.0, False),
               (1e-3, 0.0, 0.0, 0.0, 0.01, False)):
        announce("adam late", step, hp)
        want = oracle.adam_step(p, gr, m, v, *hp[:5], step, hp[5])
        pd, md, vd = dev(p), dev(m), dev(v)
        rp.adam_step(pd, dev(gr), md, vd, *hp[:5], step, hp[5])
        for got, w, what in zip((pd, md, vd), want, "pmv"):
            assert_bits_equal(host(got), w, f"{what} step={step} hp={hp}")


def test_adam_misaligned_views(rp):
    g = inputs.rng(701)
    n = 1000
    p, gr = inputs.normal(g, (n,)), inputs.normal(g, (n,), var=1e-2)
    m, v = inputs.normal(g, (n,), var=1e-4), np.abs(inputs.normal(g, (n,), var=1e-6))
    want = oracle.adam_step(p, gr, m, v, 1e-3, weight_decay=0.01, step=3, decoupled=True)
    pad = lambda a: dev(np.concatenate([np.zeros(1, np.float32), a]))[1:]  # noqa: E731
    pd, md, vd = pad(p), pad(m), pad(v)
    announce("adam misaligned")
    rp.adam_step(pd, pad(gr), md, vd, 1e-3, weight_decay=0.01, step=3, decoupled=True)
    for got, w, what in zip((pd, md, vd), want, "pmv"):
        assert_bits_equal(host(got), w, f"misaligned {what}")


# --------------------------------------------------------------------------
# Signed zeros in the product chains.  fma(a, b, q) with a negative product
# below half the smallest subnormal gives -0; masked and absent terms take no
# operation in the row order, so a chain that holds -0 keeps it, and the row
# sum of -0 chains is -0.  A kernel that padded absent terms with
# fma(+0, +0, q) would turn those chains into +0 and change outputs that take
# the sum's sign (dy = -0 minus the sum).  The parameter gradients' single
# block is still added into the +0 accumulator (+0 + (-0) = +0).
# --------------------------------------------------------------------------

def _lane_terms(cols):
    """Per column j: (t, number of terms of lane j mod 64)."""
    j = np.arange(cols)
    t = j // 64
    n = (cols - (j % 64) + 63) // 64
    return t, n


def softmax_negzero_case(rows, cols, period):
    """Y = 2^-140; dY = -2^-20 (products -2^-160 round to -0), except the last
    term of every lane that has two or more, which is -0.0 (the product with
    -0 keeps a -0 chain).  Causal rows get the pattern over their valid prefix."""
    Y = np.full((rows, cols), 2.0 ** -140, np.float32)
    dY = np.full((rows, cols), -(2.0 ** -20), np.float32)
    for r in range(rows):
        valid = cols if period == 0 else min(cols, r % period + 1)
        t, n = _lane_terms(valid)
        last = (t == n - 1) & (n >= 2)
        dY[r, :valid][last] = -0.0
    return Y, dY


@pytest.mark.parametrize("cols,period", [(65, 0), (100, 0), (130, 0), (1000, 0), (2100, 0),
                                         (3000, 0), (5000, 0), (300, 200), (1024, 1024)])
def test_softmax_backward_negative_zero_chains(rp, cols, period):
    rows = 40 if period == 0 else period
    Y, dY = softmax_negzero_case(rows, cols, period)
    want = oracle.softmax_backward_rows(Y, dY, causal_period=period)
    # the witness bites: dy = -0 minus a -0 sum is +0 (a +0 sum would give -0)
    full = min(cols, (rows - 1) % period + 1) if period else cols
    r_full = rows - 1
    cols_neg = np.nonzero(np.signbit(dY[r_full, :full]) & (dY[r_full, :full] == 0))[0]
    assert cols_neg.size and not np.signbit(want[r_full, cols_neg]).any()
    Yd, dYd = dev(Y), dev(dY)
    for name, launch in row_launches(rp, cols=cols):
        announce("softmax_backward -0 chains", cols, period, name)
        got = host(rp.softmax_backward_rows(Yd, dYd, causal_period=period, launch=launch))
        assert_bits_equal(got, want, f"{name} cols={cols} period={period}")


def norm_negzero_case(rows, cols, rms):
    """mean = 0, rstd = 1; per lane, terms in pairs (dy, x) = (+c, -tau) and
    (-c, +tau) -- products -2^-151 that round to -0, and g sums that cancel to
    +0 -- and, when a lane has an odd number of terms, a last term with
    dy = -0, x = +tau (its dx is rstd * ((-0 - a) - t b) = +0 for a -0 sum b)."""
    c, tau = 2.0 ** -81, 2.0 ** -70
    t, n = _lane_terms(cols)
    last = (n % 2 == 1) & (t == n - 1)
    dy_row = np.where(t % 2 == 0, c, -c).astype(np.float32)
    x_row = np.where(t % 2 == 0, -tau, tau).astype(np.float32)
    dy_row[last] = -0.0
    x_row[last] = tau
    X = np.repeat(x_row[None], rows, 0)
    dY = np.repeat(dy_row[None], rows, 0)
    mean = np.zeros(rows, np.float32)
    rstd = np.ones(rows, np.float32)
    return X, dY, mean, rstd, last


@pytest.mark.parametrize("rows", [50, 130])
@pytest.mark.parametrize("cols", [150, 700, 1100, 2500, 4000])
def test_layernorm_backward_negative_zero_chains(rp, rows, cols):
    X, dY, mean, rstd, last = norm_negzero_case(rows, cols, False)
    want = oracle.layernorm_backward_rows(X, dY, mean, rstd, None)
    assert last.any() and not np.signbit(want[0][:, last]).any()
    assert not np.signbit(want[1]).any()  # dgamma: -0 chains joined to +0
    for name, launch in row_launches(rp, cols=cols):
        announce("layernorm_backward -0 chains", rows, cols, name)
        got = run_lnb(rp, X, dY, mean, rstd, None, launch=launch)
        for a, b, what in zip(got, want, ("dX", "dgamma", "dbeta")):
            assert_bits_equal(a, b, f"{name} {what} rows={rows} cols={cols}")


@pytest.mark.parametrize("rows", [50, 130])
@pytest.mark.parametrize("cols", [150, 1100, 4000])
def test_rmsnorm_backward_negative_zero_chains(rp, rows, cols):
    X, dY, _, rstd, last = norm_negzero_case(rows, cols, True)
    want = oracle.rmsnorm_backward_rows(X, dY, rstd, None)
    assert last.any() and not np.signbit(want[0][:, last]).any()
    for name, launch in row_launches(rp, cols=cols):
        announce("rmsnorm_backward -0 chains", rows, cols, name)
        got = rp.rmsnorm_backward_rows(dev(X), dev(dY), dev(rstd), None, launch=launch)
        for a, b, what in zip(got, want, ("dX", "dgamma")):
            assert_bits_equal(host(a), b, f"{name} {what} rows={rows} cols={cols}")

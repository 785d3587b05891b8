"""GPU parity of the Llama-block operators against the CPU oracle (0 ULP):
sin/cos (all 2^32 inputs), the rotary embedding, RMSNorm forward and backward,
SiLU and the SiLU-gated unit forward and backward (all 2^32 gate values) --
ragged shapes, every row order, several contraction block lengths, in-place
calls, padded leading dimensions, every launch configuration and the Llama
attention / feed-forward shapes."""
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


def row_launches(rp, cols, wave_max=2048, W=64, combine=0, split=False):
    out = [("generic", rp.Launch(rp.LAUNCH_ROWS_GENERIC)), ("auto", None)]
    if W == 64 and combine == 0 and cols <= wave_max:
        out += [(f"wave{w}", rp.Launch(rp.LAUNCH_ROWS_WAVE, (w,))) for w in (1, 2, 4, 8)]
    if W == 64 and combine == 0 and split:
        # one row per workgroup, split over S waves (at most 32 values per lane)
        out += [(f"split{S}", rp.Launch(rp.LAUNCH_ROWS_WAVE, (1, S)))
                for S in (2, 4, 8) if cols <= S * 64 * 32]
    return out


def ew_launches(rp):
    return [("auto", None), ("t64", rp.Launch(rp.LAUNCH_ELEMENTWISE, (64, 0))),
            ("t1024", rp.Launch(rp.LAUNCH_ELEMENTWISE, (1024, 0))),
            ("t256b7", rp.Launch(rp.LAUNCH_ELEMENTWISE, (256, 7)))]


def inv_freq(head_dim, base=500000.0):
    return (base ** (-np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)).astype(np.float32)


# --------------------------------------------------------------------------
# sin / cos
# --------------------------------------------------------------------------

def test_sincos_ranges_and_launches(rp):
    g = inputs.rng(800)
    x = np.concatenate([inputs.uniform(g, (300000,), -4, 4),
                        inputs.uniform(g, (300000,), -2.0 ** 17, 2.0 ** 17),
                        inputs.uniform(g, (1001,), -1e30, 1e30),
                        np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45,
                                  np.float32(np.pi / 2), np.float32(np.pi), 3.4e38], np.float32)])
    ws, wc = oracle.sincos(x)
    for name, launch in ew_launches(rp):
        announce("sincos", name)
        s, c = rp.sincos(dev(x), launch=launch)
        assert_bits_equal(host(s), ws, f"sin {name}")
        assert_bits_equal(host(c), wc, f"cos {name}")


def test_sincos_exhaustive_all_bit_patterns(rp):
    import torch
    chunk = 1 << 28
    for c in range(16):
        announce("sincos exhaustive chunk", c)
        base = c * chunk
        x = (torch.arange(base, base + chunk, dtype=torch.int64, device="cuda:0")
             .to(torch.int32).view(torch.float32))
        s, co = rp.sincos(x)
        xs = (np.arange(base, base + chunk, dtype=np.uint64).astype(np.uint32)).view(np.float32)
        ws, wc = oracle.sincos(xs)
        assert_bits_equal(host(s), ws, f"sin chunk {c}")
        assert_bits_equal(host(co), wc, f"cos chunk {c}")
        del x, s, co, xs, ws, wc


# --------------------------------------------------------------------------
# rotary embedding
# --------------------------------------------------------------------------

ROPE_SHAPES = [(75, 3, 64, 0, 0), (130, 4, 128, 50, 7), (33, 1, 6, 0, 100), (20, 2, 200, 7, 0),
               (1, 1, 2, 0, 0), (64, 8, 128, 16, 1000)]


@pytest.mark.parametrize("rows,heads,hd,period,offset", ROPE_SHAPES)
def test_rope_all_launches(rp, rows, heads, hd, period, offset):
    g = inputs.rng(810 + rows + hd)
    X = inputs.normal(g, (rows, heads * hd))
    inv = inv_freq(hd)
    for inverse in (False, True):
        want = oracle.rope(X, heads, hd, inv, period, offset, inverse)
        for name, launch in [("auto", None)] + [
                (f"wave{w}", rp.Launch(rp.LAUNCH_ROWS_WAVE, (w,))) for w in (1, 2, 4, 8)]:
            announce("rope", rows, heads, hd, period, offset, inverse, name)
            got = host(rp.rope(dev(X), heads, hd, dev(inv), period, offset, inverse,
                               launch=launch))
            assert_bits_equal(got, want, f"{name} inverse={inverse}")


def test_rope_in_place_and_padded(rp):
    import torch
    g = inputs.rng(811)
    X = inputs.normal(g, (40, 4 * 64))
    inv = inv_freq(64, 10000.0)
    want = oracle.rope(X, 4, 64, inv, 16, 3)
    announce("rope in place")
    d = dev(X)
    rp.rope(d, 4, 64, dev(inv), 16, 3, out=d)
    assert_bits_equal(host(d), want, "in place")
    announce("rope padded")
    big = torch.full((40, 300), float("nan"), device="cuda:0")
    big[:, :256] = dev(X)
    out = torch.full((40, 270), -5.0, device="cuda:0")
    rp.rope(big, 4, 64, dev(inv), 16, 3, out=out[:, :256])
    o = host(out)
    assert_bits_equal(o[:, :256], want, "padded")
    assert (o[:, 256:] == -5.0).all()


def test_rope_llama_shape(rp):
    """Q of the Llama attention block: 4 x 1024 tokens, 32 heads of 128."""
    g = inputs.rng(812)
    X = inputs.normal(g, (4096, 4096))
    inv = inv_freq(128)
    want = oracle.rope(X, 32, 128, inv, 1024, 0)
    announce("rope llama")
    assert_bits_equal(host(rp.rope(dev(X), 32, 128, dev(inv), 1024, 0)), want, "llama")


# --------------------------------------------------------------------------
# RMSNorm
# --------------------------------------------------------------------------

COLS = [1, 2, 63, 64, 65, 100, 768, 1000, 2048, 2049, 4096, 5000, 8192, 16384]


@pytest.mark.parametrize("cols", COLS)
def test_rmsnorm_forward_all_launches(rp, cols):
    g = inputs.rng(820 + cols)
    X = inputs.normal(g, (75, cols), var=2.0)
    gam = 1 + inputs.normal(g, (cols,), var=0.01)
    for gamma in (gam, None):
        want, wr = oracle.rmsnorm_rows(X, gamma, eps=1e-6, with_stats=True)
        for name, launch in row_launches(rp, cols, wave_max=4096, split=True):
            announce("rmsnorm", cols, gamma is None, name)
            import torch
            r = torch.empty(75, device="cuda:0")
            got = rp.rmsnorm_rows(dev(X), None if gamma is None else dev(gamma), eps=1e-6,
                                  launch=launch, rstd_out=r)
            assert_bits_equal(host(got), want, f"{name} y")
            assert_bits_equal(host(r), wr, f"{name} rstd")


@pytest.mark.parametrize("W,combine", [(1, 0), (16, 0), (1024, 0), (64, 1), (8, 1)])
def test_rmsnorm_other_orders(rp, W, combine):
    g = inputs.rng(830 + W + combine)
    X = inputs.normal(g, (40, 777))
    want = oracle.rmsnorm_rows(X, None, row_width=W, row_combine=combine)
    announce("rmsnorm order", W, combine)
    got = rp.rmsnorm_rows(dev(X), order=rp.Order(row_width=W, row_combine=combine))
    assert_bits_equal(host(got), want, f"W={W} combine={combine}")


def rms_case(seed, rows, cols, with_gamma=True):
    g = inputs.rng(seed)
    X = inputs.normal(g, (rows, cols), var=2.0)
    gamma = (1 + inputs.normal(g, (cols,), var=0.01)) if with_gamma else None
    _, rstd = oracle.rmsnorm_rows(X, gamma, with_stats=True)
    dY = inputs.normal(g, (rows, cols), var=1e-2)
    return X, dY, rstd, gamma


@pytest.mark.parametrize("cols", COLS)
def test_rmsnorm_backward_all_launches(rp, cols):
    for rows, with_gamma in ((75, True), (130, False)):
        X, dY, rstd, gamma = rms_case(840 + cols + rows, rows, cols, with_gamma)
        want = oracle.rmsnorm_backward_rows(X, dY, rstd, gamma)
        for name, launch in row_launches(rp, cols, split=True):
            announce("rmsnorm_backward", rows, cols, with_gamma, name)
            dx, dg = rp.rmsnorm_backward_rows(dev(X), dev(dY), dev(rstd),
                                              None if gamma is None else dev(gamma),
                                              launch=launch)
            assert_bits_equal(host(dx), want[0], f"{name} dX")
            assert_bits_equal(host(dg), want[1], f"{name} dgamma")


@pytest.mark.parametrize("W,combine,k_block", [(16, 0, 0), (64, 1, 128), (8, 1, 1), (64, 0, 7),
                                               (64, 0, 0)])
def test_rmsnorm_backward_other_orders(rp, W, combine, k_block):
    X, dY, rstd, gamma = rms_case(850 + W + k_block, 150, 777)
    want = oracle.rmsnorm_backward_rows(X, dY, rstd, gamma, row_width=W, row_combine=combine,
                                        k_block=k_block)
    announce("rmsnorm_backward order", W, combine, k_block)
    dx, dg = rp.rmsnorm_backward_rows(dev(X), dev(dY), dev(rstd), dev(gamma),
                                      order=rp.Order(row_width=W, row_combine=combine,
                                                     k_block=k_block))
    assert_bits_equal(host(dx), want[0], "dX")
    assert_bits_equal(host(dg), want[1], "dgamma")


def test_rmsnorm_backward_in_place_and_llama_shape(rp):
    X, dY, rstd, gamma = rms_case(860, 200, 300)
    want = oracle.rmsnorm_backward_rows(X, dY, rstd, gamma)
    announce("rmsnorm_backward in place")
    d = dev(dY)
    dx, dg = rp.rmsnorm_backward_rows(dev(X), d, dev(rstd), dev(gamma), dx_out=d)
    assert_bits_equal(host(d), want[0], "dX = dY")
    assert_bits_equal(host(dg), want[1], "dgamma")
    X, dY, rstd, gamma = rms_case(861, 4096, 4096)
    want = oracle.rmsnorm_backward_rows(X, dY, rstd, gamma)
    announce("rmsnorm_backward llama 4096x4096")
    dx, dg = rp.rmsnorm_backward_rows(dev(X), dev(dY), dev(rstd), dev(gamma))
    assert_bits_equal(host(dx), want[0], "llama dX")
    assert_bits_equal(host(dg), want[1], "llama dgamma")


# --------------------------------------------------------------------------
# SiLU / SwiGLU
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 3, 4, 5, 1000, 1001, 4096 * 14336 // 16 + 3])
def test_silu_swiglu_all_launches(rp, n):
    g = inputs.rng(870 + n % 1000)
    G = inputs.normal(g, (n,), var=9.0)
    Uv = inputs.normal(g, (n,))
    dY = inputs.normal(g, (n,), var=1e-2)
    ws, wy = oracle.silu(G), oracle.swiglu(G, Uv)
    wdg, wdu = oracle.swiglu_backward(G, Uv, dY)
    Gd, Ud, Dd = dev(G), dev(Uv), dev(dY)
    for name, launch in ew_launches(rp):
        announce("silu/swiglu", n, name)
        assert_bits_equal(host(rp.silu(Gd, launch=launch)), ws, f"silu {name}")
        assert_bits_equal(host(rp.swiglu(Gd, Ud, launch=launch)), wy, f"swiglu {name}")
        dg, du = rp.swiglu_backward(Gd, Ud, Dd, launch=launch)
        assert_bits_equal(host(dg), wdg, f"dgate {name}")
        assert_bits_equal(host(du), wdu, f"dup {name}")
    if n > 4:
        announce("swiglu misaligned", n)
        pad = lambda a: dev(np.concatenate([np.zeros(1, np.float32), a]))[1:]  # noqa: E731
        assert_bits_equal(host(rp.swiglu(pad(G), pad(Uv))), wy, "misaligned swiglu")
        dg, du = rp.swiglu_backward(pad(G), pad(Uv), pad(dY))
        assert_bits_equal(host(dg), wdg, "misaligned dgate")


def test_swiglu_in_place(rp):
    g = inputs.rng(871)
    G, Uv, dY = inputs.normal(g, (777,)), inputs.normal(g, (777,)), inputs.normal(g, (777,))
    wy = oracle.swiglu(G, Uv)
    wdg, wdu = oracle.swiglu_backward(G, Uv, dY)
    announce("swiglu in place")
    Gd, Ud = dev(G), dev(Uv)
    rp.swiglu(Gd, Ud, out=Gd)
    assert_bits_equal(host(Gd), wy, "y = G")
    Gd, Ud, Dd = dev(G), dev(Uv), dev(dY)
    rp.swiglu_backward(Gd, Ud, Dd, dg_out=Gd, du_out=Ud)
    assert_bits_equal(host(Gd), wdg, "dG = G")
    assert_bits_equal(host(Ud), wdu, "dUp = Up")


def test_silu_and_grad_exhaustive(rp):
    """All 2^32 gate values with up = dy = 1: dG is silu'(g) and dUp is silu(g)
    exactly (RN(1 * 1) = 1, RN(1 * v) = v), so one pass covers SiLU and its
    derivative bit for bit."""
    import torch
    chunk = 1 << 28
    for c in range(16):
        announce("silu exhaustive chunk", c)
        base = c * chunk
        x = (torch.arange(base, base + chunk, dtype=torch.int64, device="cuda:0")
             .to(torch.int32).view(torch.float32))
        ones = torch.ones_like(x)
        dg, du = rp.swiglu_backward(x, ones, ones)
        xs = (np.arange(base, base + chunk, dtype=np.uint64).astype(np.uint32)).view(np.float32)
        o = np.ones_like(xs)
        wdg, wdu = oracle.swiglu_backward(xs, o, o)
        assert_bits_equal(host(dg), wdg, f"silu' chunk {c}")
        assert_bits_equal(host(du), wdu, f"silu chunk {c}")
        del x, ones, dg, du, xs, o, wdg, wdu

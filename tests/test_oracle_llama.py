"""Pins for the oracle's Llama-block operators (no GPU): sin/cos, the rotary
embedding, RMSNorm (forward and backward) and SiLU / SwiGLU (forward and
backward).

Each function is held to what the mathematics fixes independently of the
oracle: constants against their definitions at high precision, accuracy
against float64 / mpmath, exact symmetries, special values, closed forms of
constructed inputs, finite-difference checks of the float64 derivative
formulas, order witnesses and integer-exact sums.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import exactfp
import oracle
from bitcmp import assert_bits_equal
from paper_2502_19405_amd import inputs

U = 2.0 ** -24


# --------------------------------------------------------------------------
# sin / cos
# --------------------------------------------------------------------------

def check_sincos_constants(src):
    """Reduction constants and Taylor coefficients, read from the oracle
    source, equal their definitions rounded to binary32 (computed at 300
    bits)."""
    import mpmath
    mpmath.mp.prec = 300

    def lit(name):
        line = [l for l in src.splitlines() if f" {name} =" in l][0]
        return float.fromhex(line.split("=")[1].split(";")[0].strip().rstrip("f"))

    def rn(v):
        return exactfp.rn32(Fraction(mpmath.nstr(v, 90)))

    p1 = rn(mpmath.pi / 2)
    p2 = rn(mpmath.pi / 2 - p1)
    p3 = rn(mpmath.pi / 2 - p1 - mpmath.mpf(p2))
    assert lit("SC_TWO_OVER_PI") == rn(2 / mpmath.pi)
    assert (lit("SC_P1"), lit("SC_P2"), lit("SC_P3")) == (p1, p2, p3)
    for k in (3, 5, 7, 9):
        assert lit(f"SC_S{k}") == rn(mpmath.mpf((-1) ** ((k - 1) // 2)) / mpmath.factorial(k)), k
    for k in (2, 4, 6, 8, 10):
        assert lit(f"SC_C{k}") == rn(mpmath.mpf((-1) ** (k // 2)) / mpmath.factorial(k)), k


def test_sincos_constants_match_definitions():
    check_sincos_constants(open(os.path.join(os.path.dirname(oracle.__file__),
                                             "repops_ref.c")).read())


def test_sincos_special_values(ref):
    s, c = oracle.sincos1(0.0, lib=ref)
    assert s == 0 and not np.signbit(s) and c == 1
    s, c = oracle.sincos1(-0.0, lib=ref)
    assert s == 0 and np.signbit(s) and c == 1
    for v in (np.inf, -np.inf, np.nan):
        s, c = oracle.sincos1(v, lib=ref)
        assert np.isnan(s) and np.isnan(c)
    tiny = np.float32(1e-30)
    assert oracle.sincos1(tiny, lib=ref) == (tiny, np.float32(1))
    # x = RN(pi/2): sin is the nearest float to 1 - tiny, cos ~ -4.37e-8
    s, c = oracle.sincos1(np.float32(np.pi / 2), lib=ref)
    assert s == 1 and abs(c - math.cos(float(np.float32(np.pi / 2)))) < 1e-14


def ulps(err, want):
    return err / np.spacing(np.abs(want).astype(np.float32)).astype(np.float64)


@pytest.mark.parametrize("lim", [1.0, 16.0, 4096.0, 2.0 ** 17])
def test_sincos_accuracy(ref, lim):
    """|error| <= 1.5 * 2^-24 absolute and <= 2 ulp where |f| >= 2^-8 (measured
    maxima 1.17 * 2^-24 and 1.49 ulp over |x| <= 2^17)."""
    g = inputs.rng(200 + int(math.log2(lim)))
    x = inputs.uniform(g, (1_000_000,), -lim, lim)
    s, c = oracle.sincos(x, lib=ref)
    x64 = x.astype(np.float64)
    for got, want in ((s, np.sin(x64)), (c, np.cos(x64))):
        err = np.abs(got - want)
        assert err.max() <= 1.5 * U
        big = np.abs(want) >= 2.0 ** -8
        assert ulps(err[big], want[big]).max() <= 2.0


def test_sincos_near_multiples_of_half_pi(ref):
    """Arguments next to k pi/2 leave a tiny reduced argument whose relative
    accuracy needs all three parts of pi/2: within 2 ulp of mpmath there."""
    import mpmath
    mpmath.mp.prec = 200
    ks = np.unique(np.concatenate([np.arange(1, 400), inputs.rng(210).integers(400, 80000, 400)]))
    xs = []
    for k in ks:
        v = np.float32(float(k * mpmath.pi / 2))
        xs += [v, np.nextafter(v, np.float32(np.inf)), np.nextafter(v, np.float32(-np.inf))]
    x = np.array(xs, np.float32)
    s, c = oracle.sincos(x, lib=ref)
    for got, fn in ((s, mpmath.sin), (c, mpmath.cos)):
        want = np.array([float(fn(mpmath.mpf(float(v)))) for v in x])
        assert ulps(np.abs(got - want), want).max() <= 2.0


def test_sincos_symmetry_is_exact(ref):
    """sin(-x) = -sin(x) and cos(-x) = cos(x) bit for bit (rint is symmetric,
    the reduction and polynomials are odd/even, the quadrant table maps n and
    -n consistently)."""
    g = inputs.rng(211)
    x = np.concatenate([inputs.uniform(g, (200000,), 0, 2.0 ** 17),
                        inputs.uniform(g, (200000,), 0, 8)])
    s, c = oracle.sincos(x, lib=ref)
    sn, cn = oracle.sincos(-x, lib=ref)
    assert_bits_equal(sn, -s, "odd")
    assert_bits_equal(cn, c, "even")


def test_sincos_pythagoras(ref):
    g = inputs.rng(212)
    x = inputs.uniform(g, (500000,), -2.0 ** 16, 2.0 ** 16)
    s, c = oracle.sincos(x, lib=ref)
    s64, c64 = s.astype(np.float64), c.astype(np.float64)
    assert np.abs(s64 * s64 + c64 * c64 - 1).max() <= 4 * U


# --------------------------------------------------------------------------
# rotary embedding
# --------------------------------------------------------------------------

def llama_inv_freq(head_dim, base=500000.0):
    """Frequency table theta_i = base^(-2i/d) rounded to binary32 (a model input,
    like a weight)."""
    return (base ** (-np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)).astype(np.float32)


def test_rope_position_zero_is_identity(ref):
    g = inputs.rng(220)
    X = inputs.normal(g, (1, 4 * 64))
    Y = oracle.rope(X, 4, 64, llama_inv_freq(64), lib=ref)
    assert_bits_equal(Y, X, "position 0")


def test_rope_pairs_rotate_half(ref):
    """A one-hot input at column i of a head lands only at i and i + d/2 (or
    i - d/2) of the same head: the pairing is rotate-half."""
    hd, heads = 16, 2
    inv = llama_inv_freq(hd, 10000.0)
    for col in (0, 3, 8, 13, 16 + 5, 16 + 12):
        X = np.zeros((7, heads * hd), np.float32)
        X[:, col] = 1.0
        Y = oracle.rope(X, heads, hd, inv, lib=ref)
        h, i = divmod(col, hd)
        partner = h * hd + (i + hd // 2) % hd
        nz = set(np.flatnonzero(np.abs(Y).sum(0)))
        assert nz <= {col, partner} and col in nz


def test_rope_rotation_accuracy_and_inverse(ref):
    """Against the exact rotation by the float64 angle p * theta_i (with theta_i
    the binary32 table): a few ulp of the pair norm; and the inverse rotation
    undoes the forward within the same order of error."""
    g = inputs.rng(221)
    rows, heads, hd = 300, 4, 128
    inv = llama_inv_freq(hd)
    X = inputs.normal(g, (rows, heads * hd))
    Y = oracle.rope(X, heads, hd, inv, period=100, offset=7, lib=ref)
    pos = (np.arange(rows) % 100 + 7).astype(np.float64)
    ang = pos[:, None] * inv.astype(np.float64)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    X64 = X.astype(np.float64).reshape(rows, heads, hd)
    x1, x2 = X64[..., :hd // 2], X64[..., hd // 2:]
    y1 = x1 * c[:, None, :] - x2 * s[:, None, :]
    y2 = x2 * c[:, None, :] + x1 * s[:, None, :]
    want = np.concatenate([y1, y2], axis=-1).reshape(rows, heads * hd)
    norm = np.sqrt(x1 ** 2 + x2 ** 2)
    nrm = np.concatenate([norm, norm], axis=-1).reshape(rows, heads * hd)
    # angle rounding (|p theta| u) moves the point by up to |p theta| u * norm
    amp = np.concatenate([ang, ang], axis=-1)[:, None, :].repeat(heads, 1).reshape(rows, -1)
    assert (np.abs(Y - want) <= (6 + amp) * U * nrm).all()
    Z = oracle.rope(Y, heads, hd, inv, period=100, offset=7, inverse=True, lib=ref)
    assert (np.abs(Z - X) <= 12 * U * nrm).all()


def test_rope_period_and_offset(ref):
    g = inputs.rng(222)
    X = inputs.normal(g, (64, 2 * 32))
    inv = llama_inv_freq(32)
    full = oracle.rope(np.tile(X[:16], (4, 1)), 2, 32, inv, period=16, offset=3, lib=ref)
    for b in range(4):
        assert_bits_equal(full[16 * b:16 * (b + 1)],
                          oracle.rope(X[:16], 2, 32, inv, offset=3, lib=ref), f"batch {b}")


# --------------------------------------------------------------------------
# RMSNorm
# --------------------------------------------------------------------------

def rms64(x, gamma, eps):
    r = 1 / np.sqrt((x * x).mean(-1, keepdims=True) + eps)
    return x * r * gamma


def rms_vjp64(x, gamma, dy, eps):
    r = 1 / np.sqrt((x * x).mean(-1, keepdims=True) + eps)
    t = x * r
    g = dy * gamma
    return r * (g - t * (g * t).mean(-1, keepdims=True))


def test_rmsnorm_vjp_formula_is_the_gradient():
    g = inputs.rng(230)
    x = g.standard_normal(11)
    gamma = 1 + 0.1 * g.standard_normal(11)
    dy = g.standard_normal(11)
    h = 1e-6
    fd = np.array([(np.dot(rms64(x + h * e, gamma, 1e-5), dy) -
                    np.dot(rms64(x - h * e, gamma, 1e-5), dy)) / (2 * h) for e in np.eye(11)])
    assert np.allclose(fd, rms_vjp64(x, gamma, dy, 1e-5), atol=1e-7)


def test_rmsnorm_constant_rows(ref):
    """x = a (a power of two) with eps = 0: ms = a^2, rstd = 1/|a| exactly,
    y = sign(a) * gamma exactly."""
    X = np.array([[4.0] * 100, [-0.25] * 100, [2.0 ** -60] * 100], np.float32)
    gam = inputs.normal(inputs.rng(231), (100,))
    Y, rstd = oracle.rmsnorm_rows(X, gam, eps=0.0, lib=ref, with_stats=True)
    assert list(rstd) == [0.25, 4.0, 2.0 ** 60]
    assert_bits_equal(Y, np.sign(X[:, :1]) * gam[None, :], "constant rows")


@pytest.mark.parametrize("W,combine", [(64, 0), (16, 0), (64, 1), (1, 0)])
def test_rmsnorm_bound(ref, W, combine):
    g = inputs.rng(232 + W)
    X = inputs.normal(g, (64, 4096))
    gam = 1 + inputs.normal(g, (4096,), var=0.01)
    Y = oracle.rmsnorm_rows(X, gam, eps=1e-5, row_width=W, row_combine=combine, lib=ref)
    want = rms64(X.astype(np.float64), gam.astype(np.float64), float(np.float32(1e-5)))
    n = 4096
    rel = (0.5 * (n / W + math.log2(W) + 3) + 5) * U
    assert (np.abs(Y - want) <= rel * np.abs(want) + 2.0 ** -140).all()


def test_rmsnorm_gamma_none_equals_ones(ref):
    X = inputs.normal(inputs.rng(233), (9, 300))
    assert_bits_equal(oracle.rmsnorm_rows(X, None, lib=ref),
                      oracle.rmsnorm_rows(X, np.ones(300, np.float32), lib=ref), "gamma")


def test_rmsnorm_backward_bound(ref):
    g = inputs.rng(234)
    X = inputs.normal(g, (48, 2048))
    gam = 1 + inputs.normal(g, (2048,), var=0.01)
    dY = inputs.normal(g, X.shape)
    _, rstd = oracle.rmsnorm_rows(X, gam, eps=1e-5, lib=ref, with_stats=True)
    dX, dg = oracle.rmsnorm_backward_rows(X, dY, rstd, gam, lib=ref)
    want = rms_vjp64(X.astype(np.float64), gam.astype(np.float64), dY.astype(np.float64),
                     float(np.float32(1e-5)))
    scale = np.abs(dY * gam).max(axis=1, keepdims=True) * rstd[:, None]
    assert (np.abs(dX - want) <= 128 * U * scale).all()
    t64 = X.astype(np.float64) * rstd[:, None]
    dg_want = (dY.astype(np.float64) * t64).sum(0)
    nr = X.shape[0]
    gm = (64 + nr / 64 + 2) * U
    assert (np.abs(dg - dg_want) <= gm * (np.abs(dY) * np.abs(t64)).sum(0) + 1e-30).all()


def test_rmsnorm_dgamma_order_witness_and_integers(ref):
    """X = 1, eps = 0 make t = 1 exactly, so dgamma is the blocked left-to-right
    column sum of dy: 2^24 in row 0 and ones in rows 64..127 give 2^24 + 64
    with blocks of 64 and 2^24 unblocked; integer dy sums exactly."""
    rows, cols = 128, 5
    X = np.ones((rows, cols), np.float32)
    _, rstd = oracle.rmsnorm_rows(X, eps=0.0, lib=ref, with_stats=True)
    assert (rstd == 1).all()
    dY = np.zeros((rows, cols), np.float32)
    dY[0] = 2.0 ** 24
    dY[64:] = 1.0
    _, dg = oracle.rmsnorm_backward_rows(X, dY, rstd, want_dx=False, lib=ref)
    assert (dg == np.float32(2 ** 24 + 64)).all()
    _, dg0 = oracle.rmsnorm_backward_rows(X, dY, rstd, want_dx=False, k_block=0, lib=ref)
    assert (dg0 == np.float32(2 ** 24)).all()
    dYi = inputs.integers(inputs.rng(235), (rows, cols), -50, 50)
    _, dgi = oracle.rmsnorm_backward_rows(X, dYi, rstd, want_dx=False, lib=ref)
    assert np.array_equal(dgi, dYi.astype(np.int64).sum(0).astype(np.float32))


# --------------------------------------------------------------------------
# SiLU / SwiGLU
# --------------------------------------------------------------------------

def silu64(x):
    with np.errstate(over="ignore"):
        return x / (1 + np.exp(-x))


def silu_grad64(x):
    with np.errstate(over="ignore"):
        s = 1 / (1 + np.exp(-x))
    return s + x * s * (1 - s)


def test_silu_grad_formula_is_the_derivative():
    x = np.linspace(-20, 20, 4001)
    h = 1e-6
    assert np.allclose((silu64(x + h) - silu64(x - h)) / (2 * h), silu_grad64(x), atol=1e-8)


def test_silu_special_values(ref):
    assert oracle.silu1(0.0, lib=ref) == 0
    assert oracle.silu1(100.0, lib=ref) == 100
    v = oracle.silu1(-200.0, lib=ref)  # exp overflows: x / inf = -0
    assert v == 0 and np.signbit(v)
    assert oracle.silu_grad1(0.0, lib=ref) == 0.5
    assert oracle.silu_grad1(100.0, lib=ref) == 1
    assert np.isnan(oracle.silu1(np.nan, lib=ref))


def test_silu_and_grad_bounds(ref):
    """silu: relative error <= 4u (the argument -x is exact, exp_rep adds < 1
    ulp, then one rounding each for 1 + e and the division; measured maximum
    2.8u).  silu': relative to s + |x s (1 - s)|, <= (8 + 2|x|) u, the |x| from
    the cancellation in 1 - s."""
    g = inputs.rng(240)
    x = np.concatenate([inputs.uniform(g, (400000,), -30, 30), inputs.normal(g, (400000,))])
    x64 = x.astype(np.float64)
    y = oracle.silu(x, lib=ref)
    want = silu64(x64)
    assert (np.abs(y - want) <= 4 * U * np.abs(want) + 2.0 ** -140).all()
    gr = np.array([oracle.silu_grad1(v, lib=ref) for v in x[::40]], np.float64)
    xg = x64[::40]
    s = 1 / (1 + np.exp(-xg))
    mag = s + np.abs(xg * s * (1 - s))
    assert (np.abs(gr - silu_grad64(xg)) <= (8 + 2 * np.abs(xg)) * U * mag).all()


def test_swiglu_forward_and_backward(ref):
    g = inputs.rng(241)
    G = inputs.normal(g, (100000,), var=4.0)
    Uv = inputs.normal(g, (100000,))
    dY = inputs.normal(g, (100000,), var=1e-2)
    y = oracle.swiglu(G, Uv, lib=ref)
    # one more rounding than silu: the product with u
    s = oracle.silu(G, lib=ref)
    assert_bits_equal(y, s * Uv, "swiglu = RN(silu(g) u)")
    dg, du = oracle.swiglu_backward(G, Uv, dY, lib=ref)
    assert_bits_equal(du, dY * s, "dup = RN(dy silu(g))")
    G64, U64, D64 = (a.astype(np.float64) for a in (G, Uv, dY))
    want = D64 * U64 * silu_grad64(G64)
    sg = 1 / (1 + np.exp(-G64))
    mag = np.abs(D64 * U64) * (sg + np.abs(G64 * sg * (1 - sg)))
    assert (np.abs(dg - want) <= (10 + 2 * np.abs(G64)) * U * mag + 2.0 ** -140).all()

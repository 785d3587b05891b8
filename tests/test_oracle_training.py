"""Pins for the oracle's training-step operators (no GPU): softmax, LayerNorm
and GELU backward, and the Adam / AdamW step.

Each derivative is pinned twice: its float64 formula is first checked against
central finite differences of the float64 forward (so the formula really is
the gradient), then the binary32 oracle is held to an error bound around that
formula.  Closed forms, order witnesses and special cases pin the bits where
the arithmetic allows it.
"""
import math
import os

import numpy as np
import pytest

import exactfp
import oracle
from bitcmp import assert_bits_equal
from paper_2502_19405_amd import inputs

U = 2.0 ** -24
GC = float(np.float32(0.044715))
SQ = float(np.float32(math.sqrt(2 / math.pi)))


# --------------------------------------------------------------------------
# softmax backward
# --------------------------------------------------------------------------

def softmax64(x):
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def softmax_vjp64(y, dy):
    return y * (dy - (y * dy).sum(axis=-1, keepdims=True))


def test_softmax_vjp_formula_is_the_gradient():
    g = inputs.rng(100)
    x = g.standard_normal(7) * 2
    dy = g.standard_normal(7)
    h = 1e-6
    fd = np.array([(np.dot(softmax64(x + h * e), dy) - np.dot(softmax64(x - h * e), dy)) / (2 * h)
                   for e in np.eye(7)])
    assert np.allclose(fd, softmax_vjp64(softmax64(x), dy), atol=1e-8)


def test_softmax_backward_one_hot_closed_form(ref):
    """dy = e_m: the fixed-order sum is y_m exactly (every other term adds +0),
    so dx_j = RN(y_j * RN(0 - y_m)) and dx_m = RN(y_m * RN(1 - y_m))."""
    g = inputs.rng(101)
    Y = oracle.softmax_rows(inputs.normal(g, (5, 300), var=4.0), lib=ref)
    for m in (0, 17, 299):
        dY = np.zeros_like(Y)
        dY[:, m] = 1.0
        dX = oracle.softmax_backward_rows(Y, dY, lib=ref)
        want = Y * (np.float32(0) - Y[:, m:m + 1])
        want[:, m] = Y[:, m] * (np.float32(1) - Y[:, m])
        assert_bits_equal(dX, want.astype(np.float32), f"one-hot {m}")


@pytest.mark.parametrize("W,combine", [(64, 0), (16, 0), (64, 1)])
def test_softmax_backward_bound(ref, W, combine):
    g = inputs.rng(102 + W)
    X = inputs.normal(g, (40, 777), var=4.0)
    Y = oracle.softmax_rows(X, lib=ref)
    dY = inputs.normal(g, (40, 777))
    dX = oracle.softmax_backward_rows(Y, dY, row_width=W, row_combine=combine, lib=ref)
    Y64, dY64 = Y.astype(np.float64), dY.astype(np.float64)
    s = (Y64 * dY64).sum(axis=1, keepdims=True)
    want = Y64 * (dY64 - s)  # exact for the binary32 inputs the oracle saw
    n = 777
    gam = (n / W + math.log2(W) + 2) * U
    bound = np.abs(Y64) * (2 * U * np.abs(dY64 - s) + gam * np.abs(Y64 * dY64).sum(1, keepdims=True))
    assert (np.abs(dX - want) <= bound + 2.0 ** -140).all()


def test_softmax_backward_causal_masked_zero(ref):
    g = inputs.rng(103)
    X = inputs.normal(g, (16, 40), var=4.0)
    Y = oracle.softmax_rows(X, causal_period=8, lib=ref)
    dY = inputs.normal(g, (16, 40))
    dY_noisy = dY.copy()
    for r in range(16):
        dY_noisy[r, r % 8 + 1:] = np.nan  # masked inputs are never read
    dX = oracle.softmax_backward_rows(Y, dY_noisy, causal_period=8, lib=ref)
    for r in range(16):
        keep = r % 8 + 1
        assert (dX[r, keep:].view(np.uint32) == 0).all()
        pre = oracle.softmax_backward_rows(np.ascontiguousarray(Y[r:r + 1, :keep]),
                                           np.ascontiguousarray(dY[r:r + 1, :keep]), lib=ref)
        assert_bits_equal(dX[r, :keep], pre[0], f"row {r}")


# --------------------------------------------------------------------------
# LayerNorm backward
# --------------------------------------------------------------------------

def ln64(x, gamma, eps):
    mu = x.mean(-1, keepdims=True)
    var = ((x - mu) ** 2).mean(-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gamma


def ln_vjp64(x, gamma, dy, eps):
    n = x.shape[-1]
    mu = x.mean(-1, keepdims=True)
    rstd = 1 / np.sqrt(((x - mu) ** 2).mean(-1, keepdims=True) + eps)
    t = (x - mu) * rstd
    gdy = dy * gamma
    return rstd * (gdy - gdy.mean(-1, keepdims=True) - t * (gdy * t).mean(-1, keepdims=True))


def test_layernorm_vjp_formula_is_the_gradient():
    g = inputs.rng(110)
    x = g.standard_normal(9)
    gamma = 1 + 0.1 * g.standard_normal(9)
    dy = g.standard_normal(9)
    h = 1e-6
    fd = np.array([(np.dot(ln64(x + h * e, gamma, 1e-5), dy) -
                    np.dot(ln64(x - h * e, gamma, 1e-5), dy)) / (2 * h) for e in np.eye(9)])
    assert np.allclose(fd, ln_vjp64(x, gamma, dy, 1e-5), atol=1e-7)


def test_layernorm_backward_bound(ref):
    d = inputs.distilbert_mlp(tokens=48)
    g = inputs.rng(111)
    X = d["X"]
    dY = inputs.normal(g, X.shape)
    _, mean, rstd = oracle.layernorm_rows(X, d["gamma"], d["beta"], eps=1e-5, lib=ref,
                                          with_stats=True)
    dX, dg, db = oracle.layernorm_backward_rows(X, dY, mean, rstd, d["gamma"], lib=ref)
    want = ln_vjp64(X.astype(np.float64), d["gamma"].astype(np.float64), dY.astype(np.float64),
                    float(np.float32(1e-5)))
    scale = np.abs(dY * d["gamma"]).max(axis=1, keepdims=True) * rstd[:, None]
    assert (np.abs(dX - want) <= 256 * U * scale).all()
    # parameter gradients against float64 column sums of the forward's t
    t64 = (X.astype(np.float64) - mean[:, None]) * rstd[:, None]
    dg_want = (dY.astype(np.float64) * t64).sum(0)
    db_want = dY.astype(np.float64).sum(0)
    nr = X.shape[0]
    gam = (64 + nr / 64 + 2) * U
    assert (np.abs(dg - dg_want) <= gam * (np.abs(dY) * np.abs(t64)).sum(0) + 1e-30).all()
    assert (np.abs(db - db_want) <= gam * np.abs(dY).sum(0)).all()


def test_layernorm_param_grads_order_witness(ref):
    """dbeta_j is the blocked left-to-right sum over rows: the W1 witness on a
    column (2^24 in row 0, ones in rows 64..127) gives 2^24 + 64 with blocks of
    64 and 2^24 with one block."""
    rows, cols = 128, 3
    X = inputs.normal(inputs.rng(112), (rows, cols))
    _, mean, rstd = oracle.layernorm_rows(X, lib=ref, with_stats=True)
    dY = np.zeros((rows, cols), np.float32)
    dY[0, :] = 2.0 ** 24
    dY[64:, :] = 1.0
    _, _, db = oracle.layernorm_backward_rows(X, dY, mean, rstd, want_dx=False, lib=ref)
    assert (db == np.float32(2 ** 24 + 64)).all()
    _, _, db0 = oracle.layernorm_backward_rows(X, dY, mean, rstd, want_dx=False, k_block=0,
                                               lib=ref)
    assert (db0 == np.float32(2 ** 24)).all()


def test_layernorm_param_grads_integer_exact(ref):
    g = inputs.rng(113)
    X = inputs.normal(g, (300, 40))
    _, mean, rstd = oracle.layernorm_rows(X, lib=ref, with_stats=True)
    dY = inputs.integers(g, (300, 40), -50, 50)
    _, _, db = oracle.layernorm_backward_rows(X, dY, mean, rstd, want_dx=False, lib=ref)
    assert np.array_equal(db, dY.astype(np.int64).sum(0).astype(np.float32))


def test_layernorm_backward_gamma_none_equals_ones_for_dx(ref):
    """With gamma absent g = dy; with gamma = 1, g = dy * 1 = dy exactly: the
    input gradients agree bit for bit."""
    g = inputs.rng(114)
    X = inputs.normal(g, (10, 200))
    dY = inputs.normal(g, (10, 200))
    _, mean, rstd = oracle.layernorm_rows(X, lib=ref, with_stats=True)
    a, _, _ = oracle.layernorm_backward_rows(X, dY, mean, rstd, None, lib=ref)
    b, _, _ = oracle.layernorm_backward_rows(X, dY, mean, rstd, np.ones(200, np.float32), lib=ref)
    assert_bits_equal(a, b, "gamma None vs ones")


# --------------------------------------------------------------------------
# bias gradient (column sums)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("k_block", [64, 0, 7, 1])
def test_colsum_equals_the_contraction_with_ones(ref, k_block):
    """fma(1, y, P) rounds once, exactly as P + y: the column sums equal the
    oracle's matrix product ones^T dY bit for bit under every block length."""
    g = inputs.rng(140 + k_block)
    dY = inputs.normal(g, (300, 77))
    ones = np.ones((1, 300), np.float32)
    want = oracle.matmul(ones, dY, k_block=k_block, lib=ref)[0]
    assert_bits_equal(oracle.colsum_rows(dY, k_block, lib=ref), want, f"k_block={k_block}")


def test_colsum_witness_and_integers(ref):
    dY = np.zeros((128, 3), np.float32)
    dY[0] = 2.0 ** 24
    dY[64:] = 1.0
    assert (oracle.colsum_rows(dY, 64, lib=ref) == np.float32(2 ** 24 + 64)).all()
    assert (oracle.colsum_rows(dY, 0, lib=ref) == np.float32(2 ** 24)).all()
    dYi = inputs.integers(inputs.rng(141), (500, 9), -100, 100)
    assert np.array_equal(oracle.colsum_rows(dYi, lib=ref), dYi.astype(np.int64).sum(0).astype(np.float32))
    assert (oracle.colsum_rows(np.zeros((0, 5), np.float32), lib=ref).view(np.uint32) == 0).all()


# --------------------------------------------------------------------------
# GELU backward
# --------------------------------------------------------------------------

def gelu64(x):
    z = SQ * (x + GC * x ** 3)
    return x / (1 + np.exp(-2 * z))


def gelu_grad64(x):
    z = SQ * (x + GC * x ** 3)
    s = 1 / (1 + np.exp(-2 * z))
    return s + x * s * (1 - s) * 2 * SQ * (1 + 3 * GC * x ** 2)


def test_gelu_grad_formula_is_the_derivative():
    x = np.linspace(-8, 8, 1601)
    h = 1e-6
    fd = (gelu64(x + h) - gelu64(x - h)) / (2 * h)
    assert np.allclose(fd, gelu_grad64(x), atol=1e-8)


def test_gelu_grad_special_values(ref):
    assert oracle.gelu_grad1(0.0, lib=ref) == 0.5
    assert oracle.gelu_grad1(30.0, lib=ref) == 1.0
    z = oracle.gelu_grad1(-30.0, lib=ref)
    assert z == 0 and not np.signbit(z)


def test_gelu_grad_bound(ref):
    """Error relative to the magnitude of the two terms s and |x s (1-s) k|:
    <= (8 + 4|w|) u, w = -2z (the exp amplification as in the forward), while
    exp(w) is finite (measured maximum 2.5 (1 + |w|) u)."""
    g = inputs.rng(120)
    x = np.concatenate([inputs.uniform(g, (300000,), -12, 12), inputs.normal(g, (300000,))])
    dy = np.ones_like(x)
    got = oracle.gelu_backward(x, dy, lib=ref).astype(np.float64)
    x64 = x.astype(np.float64)
    z = SQ * (x64 + GC * x64 ** 3)
    w = -2 * z
    with np.errstate(over="ignore"):
        s = 1 / (1 + np.exp(w))
    k = 2 * SQ * (1 + float(np.float32(0.134145)) * x64 ** 2)
    want = s + x64 * s * (1 - s) * k
    mag = s + np.abs(x64 * s * (1 - s) * k)
    fin = w < 88.5
    assert (np.abs(got[fin] - want[fin]) <= (8 + 4 * np.abs(w[fin])) * U * mag[fin] + 2.0 ** -140).all()
    over = w > 88.8  # exp(w) overflows: s = +0 and the gradient is +0, true value < 2^-100
    assert over.any() and (got[over] == 0).all() and (np.abs(want[over]) < 2.0 ** -100).all()
    dy = inputs.normal(g, x.shape)
    dx = oracle.gelu_backward(x, dy, lib=ref)
    grads = np.array([oracle.gelu_grad1(v, lib=ref) for v in x[:2000]], np.float32)
    assert_bits_equal(dx[:2000], dy[:2000] * grads, "dy * gelu'")


# --------------------------------------------------------------------------
# Adam / AdamW
# --------------------------------------------------------------------------

def test_adam_scalars(ref):
    """Step scalars come from binary64 and one final rounding: within half an
    ulp (plus the binary64 steps' own error) of the exact values computed with
    mpmath, including 1 - b2^t, which cancels for small t."""
    import mpmath
    mpmath.mp.prec = 120
    lr, wd = np.float32(1e-3), np.float32(0.01)
    for b1, b2 in ((0.9, 0.999), (0.5, 0.95), (0.95, 0.9999)):
        for t in (1, 2, 3, 10, 1000, 100000):
            sc = oracle.adam_scalars(lr, b1, b2, wd, t, lib=ref)
            B1, B2 = (mpmath.mpf(float(np.float32(b))) for b in (b1, b2))
            L, D = mpmath.mpf(float(lr)), mpmath.mpf(float(wd))
            exact = [1 - B1, 1 - B2, L / (1 - B1 ** t), mpmath.sqrt(1 - B2 ** t),
                     1 - L * D, B1 ** t]
            for got, want in zip(sc, exact):
                w = float(want)
                assert abs(float(got) - w) <= 1.001 * U * abs(w) + 1e-45, (b1, b2, t)
    sc = oracle.adam_scalars(1e-3, 0.5, 0.999, 0.0, 7, lib=ref)
    assert sc[5] == np.float32(0.5 ** 7)  # powers of two are exact
    sc = oracle.adam_scalars(1e-3, 0.9, 0.999, 0.0, 1, lib=ref)
    assert sc[0] == np.float32(1) - np.float32(0.9)  # 1 - b1 (exact by Sterbenz)


def test_adam_zero_gradient_keeps_parameters(ref):
    g = inputs.rng(130)
    p = inputs.normal(g, (1000,))
    z = np.zeros_like(p)
    for decoupled in (False, True):
        p2, m2, v2 = oracle.adam_step(p, z, z, z, 1e-3, decoupled=decoupled, lib=ref)
        assert_bits_equal(p2, p, "p")
        assert (m2.view(np.uint32) == 0).all() and (v2.view(np.uint32) == 0).all()


def adam64(p, g, m, v, lr, b1, b2, eps, wd, t, decoupled):
    if wd:
        if decoupled:
            p = p * (1 - lr * wd)
        else:
            g = g + wd * p
    m = b1 * m + (1 - b1) * g
    v = b2 * v + (1 - b2) * g * g
    bc1, bc2 = 1 - b1 ** t, 1 - b2 ** t
    p = p - lr / bc1 * m / (np.sqrt(v) / np.sqrt(bc2) + eps)
    return p, m, v


@pytest.mark.parametrize("wd,decoupled", [(0.0, False), (0.01, False), (0.01, True)])
def test_adam_against_float64(ref, wd, decoupled):
    g = inputs.rng(131)
    n = 20000
    p = inputs.normal(g, (n,))
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    lr, b1, b2, eps = 1e-3, 0.9, 0.999, 1e-8
    f = [np.float32(a) for a in (lr, b1, b2, eps, wd)]
    lr64, b164, b264, eps64, wd64 = (float(a) for a in f)
    for t in range(1, 6):
        grad = inputs.normal(g, (n,), var=0.01)
        p1, m1, v1 = oracle.adam_step(p, grad, m, v, lr, b1, b2, eps, wd, t, decoupled, lib=ref)
        P, M, V = adam64(p.astype(np.float64), grad.astype(np.float64), m.astype(np.float64),
                         v.astype(np.float64), lr64, b164, b264, eps64, wd64, t, decoupled)
        # the gradient that enters the moments: coupled decay adds wd * p (one rounding)
        geff = np.abs(grad.astype(np.float64))
        if wd and not decoupled:
            geff = geff + wd64 * np.abs(p.astype(np.float64))
        dm = 4 * U * (np.abs(M) + geff * 0.1)
        assert (np.abs(m1 - M) <= dm).all()
        assert (np.abs(v1 - V) <= 6 * U * np.abs(V) + 1e-45).all()
        # p: roundings of dec and p * dec (decoupled decay) and of p - update, a
        # few u of relative error in the update term
        # lr/bc1 * m / (sqrt(v)/sqrt(bc2) + eps), and m's error (the bound
        # above) carried through the update's linear dependence on m
        upd = p.astype(np.float64) * (1 - lr64 * wd64 if decoupled else 1) - P
        carry = np.where(M != 0, np.abs(upd) / np.where(M != 0, np.abs(M), 1) * dm, 0)
        rp = 3 if (wd and decoupled) else 1
        assert (np.abs(p1 - P) <= rp * U * np.abs(P) + 8 * U * np.abs(upd) + carry).all()
        p, m, v = p1, m1, v1


def test_adam_coupled_equals_decoupled_without_decay(ref):
    g = inputs.rng(132)
    p, gr = inputs.normal(g, (500,)), inputs.normal(g, (500,))
    m, v = inputs.normal(g, (500,), 0.01), np.abs(inputs.normal(g, (500,), 0.01))
    a = oracle.adam_step(p, gr, m, v, 1e-3, step=4, decoupled=False, lib=ref)
    b = oracle.adam_step(p, gr, m, v, 1e-3, step=4, decoupled=True, lib=ref)
    for x, y in zip(a, b):
        assert_bits_equal(x, y, "coupled vs decoupled, wd = 0")


def check_training_constants(src):
    """The backward constants, read from the oracle source, equal their
    definitions rounded to binary32."""
    import mpmath
    mpmath.mp.prec = 200
    from fractions import Fraction

    def lit(name):
        line = [l for l in src.splitlines() if f" {name} =" in l][0]
        return float.fromhex(line.split("=")[1].strip().rstrip(";").rstrip("f"))

    assert lit("GELU_C3") == exactfp.rn32(Fraction("0.134145"))
    sq = exactfp.rn32(Fraction(mpmath.nstr(mpmath.sqrt(2 / mpmath.pi), 60)))
    assert lit("GELU_SQ2") == 2 * sq


def test_training_constants_match_definitions():
    check_training_constants(open(os.path.join(os.path.dirname(oracle.__file__),
                                               "repops_ref.c")).read())

"""GPU parity of repops_matmul / repops_bmm against the CPU oracle (0 ULP).

Small and ragged shapes are compared on every output; every launch
configuration (simple, each vector-tiled and each matrix-core table entry)
must give the same bits, under every transposition and order descriptor the
configuration accepts.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal
from gpu_util import announce, dev, host, same_bits
from paper_2502_19405_amd import inputs

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "order_witnesses.json")


@pytest.fixture(scope="module")
def rp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2502_19405_amd import repops
    repops.load()
    return repops


def launches(rp, k_block=64, fused=True):
    """Every launch configuration that accepts this order descriptor."""
    out = [("simple", rp.Launch(rp.LAUNCH_GEMM_SIMPLE))]
    for idx, name in enumerate(rp.gemm_configs(rp.LAUNCH_GEMM_TILED)):
        bk = int(name.split("/")[0].split("x")[2])
        if k_block == 0 or k_block % bk == 0:
            out.append((f"tiled{idx}:{name}", rp.Launch(rp.LAUNCH_GEMM_TILED, (idx,))))
    if fused:
        for idx, name in enumerate(rp.gemm_configs(rp.LAUNCH_GEMM_MFMA)):
            bk = int(name.split("/")[0].split("x")[2])
            if k_block == 0 or k_block % bk == 0:
                out.append((f"mfma{idx}:{name}", rp.Launch(rp.LAUNCH_GEMM_MFMA, (idx,))))
    return out


# Includes shapes the global-to-LDS staged kernels take (K % 16 == 0, N % 4 == 0)
# with ragged row / column edges, and shapes they decline (fallback kernels).
SHAPES = [(1, 1, 1), (7, 5, 3), (33, 17, 64), (65, 70, 130), (129, 257, 100), (200, 131, 333),
          (64, 64, 0), (96, 80, 64), (200, 132, 48), (65, 68, 256), (130, 260, 160),
          (300, 36, 1024)]
ORDERS = [(64, 0), (0, 0), (128, 0), (64, 1), (32, 1)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("k_block,k_inner", [(64, 0), (0, 0), (64, 1)])
def test_matmul_gelu_all_launches(rp, shape, k_block, k_inner):
    # H = A.B + bias and G = gelu(H) from one pass: H the oracle's product, G
    # the oracle's elementwise GELU of that product, under every launch and
    # transposition; inputs scaled so that H spans GELU's curved part.
    m, n, k = shape
    g = inputs.rng(5 * m + n + 11 * k + k_block + k_inner)
    A = (inputs.normal(g, (m, k)) * np.float32(1.5 / math.sqrt(max(k, 1)))).astype(np.float32)
    B = inputs.normal(g, (k, n))
    bias = inputs.uniform(g, (n,), -2.0, 2.0)
    want_h = oracle.matmul(A, B, bias, k_block=k_block, k_inner=k_inner)
    want_g = oracle.gelu(want_h)
    order = rp.Order(k_block=k_block, k_inner=k_inner)
    dA, dB, dbias = dev(A), dev(B), dev(bias)
    dAt, dBt = dev(np.ascontiguousarray(A.T)), dev(np.ascontiguousarray(B.T))
    for name, launch in [("auto", None)] + launches(rp, k_block, k_inner == 0):
        announce("matmul_gelu", shape, k_block, k_inner, name)
        for ta, tb in ((0, 0), (1, 1)):
            a = dAt.t() if ta else dA
            b = dBt.t() if tb else dB
            h, gl = rp.matmul_gelu(a, b, dbias, order=order, launch=launch)
            assert_bits_equal(host(h), want_h, f"{name} H trans {ta}{tb}")
            assert_bits_equal(host(gl), want_g, f"{name} G trans {ta}{tb}")
    # no bias; padded output rows (ldh, ldg > n); the separate calls give the same bits
    import torch
    Hp = torch.full((m, n + 3), float("nan"), device=dA.device)
    Gp = torch.full((m, n + 5), float("nan"), device=dA.device)
    rp.matmul_gelu(dA, dB, None, order=order, out=Hp[:, :n], gelu_out=Gp[:, :n])
    h_sep = rp.matmul(dA, dB, None, order=order)
    assert same_bits(Hp[:, :n], h_sep)
    assert same_bits(Gp[:, :n], rp.gelu(h_sep.contiguous(), order=order))
    assert torch.isnan(Hp[:, n:]).all() and torch.isnan(Gp[:, n:]).all()


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("k_block,k_inner", [(64, 0), (0, 0), (64, 1)])
def test_matmul_gelu_backward_all_launches(rp, shape, k_block, k_inner):
    # C = gelu_backward(X, A.B) from one pass: the oracle's product, then the
    # oracle's GELU backward with that product as dy, under every launch and
    # transposition; alone and as one product of a grouped call
    m, n, k = shape
    g = inputs.rng(7 * m + 3 * n + 13 * k + k_block + k_inner)
    A = inputs.normal(g, (m, k))
    B = (inputs.normal(g, (k, n)) * np.float32(0.1)).astype(np.float32)
    X = inputs.uniform(g, (m, n), -4.0, 4.0)
    want = oracle.gelu_backward(X, oracle.matmul(A, B, k_block=k_block, k_inner=k_inner))
    order = rp.Order(k_block=k_block, k_inner=k_inner)
    dA, dB, dX = dev(A), dev(B), dev(X)
    dAt, dBt = dev(np.ascontiguousarray(A.T)), dev(np.ascontiguousarray(B.T))
    for name, launch in [("auto", None)] + launches(rp, k_block, k_inner == 0):
        announce("matmul_gelu_backward", shape, k_block, k_inner, name)
        for ta, tb in ((0, 0), (1, 1)):
            a = dAt.t() if ta else dA
            b = dBt.t() if tb else dB
            got = rp.matmul_gelu_backward(a, b, dX, order=order, launch=launch)
            assert_bits_equal(host(got), want, f"{name} trans {ta}{tb}")
    import torch
    # the forward input in a padded view, and the separate calls give the same bits
    Xp = torch.full((m, n + 7), float("nan"), device=dA.device)
    Xp[:, :n] = dX
    got = rp.matmul_gelu_backward(dA, dB, Xp[:, :n], order=order)
    p = rp.matmul(dA, dB, order=order)
    assert same_bits(got, rp.gelu_backward(dX, p, order=order))
    # grouped beside a plain product: each with its own bits
    other = dev(inputs.normal(g, (k, 2 * n + 1)))
    announce("grouped gelu_backward", shape, k_block, k_inner)
    plain, gb = rp.matmul_grouped([(dA, other, None, None), (dA, dB, None, None, dX)],
                                  order=order)
    assert same_bits(plain, rp.matmul(dA, other, order=order))
    assert_bits_equal(host(gb), want, f"grouped {shape}")


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("k_block,k_inner", ORDERS)
def test_matmul_small_all_launches(rp, shape, k_block, k_inner):
    m, n, k = shape
    g = inputs.rng(m + 3 * n + 7 * k + k_block + k_inner)
    A = inputs.normal(g, (m, k))
    B = inputs.normal(g, (k, n))
    bias = inputs.uniform(g, (n,), -0.1, 0.1)
    want = oracle.matmul(A, B, bias, k_block=k_block, k_inner=k_inner)
    want_t = oracle.matmul(np.ascontiguousarray(A.T), np.ascontiguousarray(B.T), bias,
                           trans_a=True, trans_b=True, k_block=k_block, k_inner=k_inner)
    assert_bits_equal(want_t, want, "oracle layout invariance")
    order = rp.Order(k_block=k_block, k_inner=k_inner)
    dA, dB, dbias = dev(A), dev(B), dev(bias)
    dAt, dBt = dev(np.ascontiguousarray(A.T)), dev(np.ascontiguousarray(B.T))
    for name, launch in launches(rp, k_block, k_inner == 0):
        announce("matmul", shape, k_block, k_inner, name)
        got = rp.matmul(dA, dB, dbias, order=order, launch=launch)
        assert_bits_equal(host(got), want, f"{name} {shape}")
        for ta, tb in ((1, 0), (0, 1), (1, 1)):
            a = dAt.t() if ta else dA
            b = dBt.t() if tb else dB
            got_t = rp.matmul(a, b, dbias, order=order, launch=launch)
            assert_bits_equal(host(got_t), want, f"{name} trans {ta}{tb}")


def test_matmul_witnesses_on_gpu(rp):
    """The hand-derived order witnesses, through every launch configuration."""
    ws = {w["name"]: w for w in json.load(open(GOLDEN))["witnesses"]}

    def vec(spec, n):
        v = np.zeros(n, np.float32)
        for key, val in spec.items():
            lo, hi = (map(int, key.split(":")) if ":" in key else (int(key), int(key) + 1))
            v[lo:hi] = np.float32(float.fromhex(val))
        return v

    w1, w2, w3 = ws["W1_blocked_vs_sequential"], ws["W2_left_to_right_vs_pairwise"], ws["W3_fused_vs_unfused"]
    cases = [
        (vec(w1["a_nonzero"], 128), np.ones(128, np.float32), 64, 0, w1["expect"]),
        (vec(w1["a_nonzero"], 128), np.ones(128, np.float32), 0, 0, w1["wrong_order"]["expect"]),
        (vec(w2["a_nonzero"], 256), np.ones(256, np.float32), 64, 0, w2["expect"]),
        (np.array([float.fromhex(s) for s in w3["a"]], np.float32),
         np.array([float.fromhex(s) for s in w3["b"]], np.float32), 64, 0, w3["expect_fma"]),
        (np.array([float.fromhex(s) for s in w3["a"]], np.float32),
         np.array([float.fromhex(s) for s in w3["b"]], np.float32), 64, 1, w3["expect_mul_add"]),
    ]
    for a, b, kb, ki, expect in cases:
        # replicate the witness over a 70 x 70 output so every tile position sees it
        A = np.tile(a, (70, 1)).astype(np.float32)
        B = np.tile(b[:, None], (1, 70)).astype(np.float32)
        want = np.float32(float.fromhex(expect))
        for name, launch in launches(rp, kb, ki == 0):
            announce("witness", kb, ki, name)
            got = host(rp.matmul(dev(A), dev(B), order=rp.Order(k_block=kb, k_inner=ki),
                                 launch=launch))
            assert (got.view(np.uint32) == want.view(np.uint32)).all(), (name, expect)


def test_matmul_integer_exact_and_bias_null(rp):
    d = inputs.gemm2048_int(n=512)
    exact = d["A"].astype(np.float64) @ d["B"].astype(np.float64)
    for name, launch in launches(rp):
        announce("int512", name)
        got = host(rp.matmul(dev(d["A"]), dev(d["B"]), dev(d["bias"]), launch=launch))
        assert np.array_equal(got, (exact + d["bias"]).astype(np.float32)), name
        got0 = host(rp.matmul(dev(d["A"]), dev(d["B"]), None, launch=launch))
        assert np.array_equal(got0, exact.astype(np.float32)), name


def test_matmul_k_zero_gives_bias_or_plus_zero(rp):
    import torch
    A = torch.empty((5, 0), device="cuda:0")
    B = torch.empty((0, 6), device="cuda:0")
    bias = dev(np.arange(6, dtype=np.float32) - 2.5)
    announce("k=0")
    got = host(rp.matmul(A, B))
    assert (got.view(np.uint32) == 0).all()
    got_b = host(rp.matmul(A, B, bias))
    assert_bits_equal(got_b, np.broadcast_to(host(bias), (5, 6)), "k=0 bias")


def test_matmul_padded_leading_dimensions(rp):
    import torch
    g = inputs.rng(77)
    m, n, k = 45, 37, 150
    A = inputs.normal(g, (m, k)); B = inputs.normal(g, (k, n))
    want = oracle.matmul(A, B)
    Ap = torch.zeros((m, k + 9), device="cuda:0"); Ap[:, :k] = dev(A)
    Bp = torch.zeros((k, n + 5), device="cuda:0"); Bp[:, :n] = dev(B)
    Cp = torch.full((m, n + 3), float("nan"), device="cuda:0")
    for name, launch in launches(rp):
        announce("padded", name)
        rp.matmul(Ap[:, :k], Bp[:, :n], launch=launch, out=Cp[:, :n])
        got = host(Cp)
        assert_bits_equal(got[:, :n], want, name)
        assert np.isnan(got[:, n:]).all()


def test_bmm_batches_and_alpha(rp):
    g = inputs.rng(78)
    A = inputs.normal(g, (2, 3, 70, 130))
    B = inputs.normal(g, (2, 3, 130, 45))
    alpha = np.float32(1 / math.sqrt(128))
    want = oracle.bmm(A, B, alpha=alpha)
    for name, launch in launches(rp):
        announce("bmm", name)
        got = host(rp.bmm(dev(A), dev(B), alpha=float(alpha), launch=launch))
        assert_bits_equal(got, want, name)
        # transposed operands (views) give the same bits
        At = dev(np.ascontiguousarray(A.transpose(0, 1, 3, 2))).transpose(2, 3)
        Bt = dev(np.ascontiguousarray(B.transpose(0, 1, 3, 2))).transpose(2, 3)
        got_t = host(rp.bmm(At, Bt, alpha=float(alpha), launch=launch))
        assert_bits_equal(got_t, want, name + " transposed")


def test_bmm_staged_shapes(rp):
    """Batched products whose shapes the staged kernels take (k = 128, the
    attention head size), ragged rows and columns."""
    g = inputs.rng(81)
    A = inputs.normal(g, (2, 3, 70, 128))
    B = inputs.normal(g, (2, 3, 128, 44))
    want = oracle.bmm(A, B, alpha=0.125)
    Bt = np.ascontiguousarray(B.transpose(0, 1, 3, 2))
    for name, launch in launches(rp):
        announce("bmm staged", name)
        assert_bits_equal(host(rp.bmm(dev(A), dev(B), alpha=0.125, launch=launch)), want, name)
        got_t = rp.bmm(dev(A), dev(Bt).transpose(2, 3), alpha=0.125, launch=launch)
        assert_bits_equal(host(got_t), want, name + " trans_b")


def test_bmm_batch_one_equals_matmul_and_loop(rp):
    g = inputs.rng(79)
    A = inputs.normal(g, (1, 1, 90, 200))
    B = inputs.normal(g, (1, 1, 200, 66))
    dA, dB = dev(A), dev(B)
    announce("bmm batch 1 vs matmul")
    assert same_bits(rp.bmm(dA, dB)[0, 0], rp.matmul(dA[0, 0], dB[0, 0]))


def test_determinism_run_to_run_and_streams(rp):
    import torch
    g = inputs.rng(80)
    A = dev(inputs.normal(g, (300, 500)))
    B = dev(inputs.normal(g, (500, 400)))
    announce("determinism")
    first = rp.matmul(A, B)
    for _ in range(3):
        assert same_bits(rp.matmul(A, B), first)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        other = rp.matmul(A, B)
    s.synchronize()
    assert same_bits(other, first)


def _adversarial(mode, g, m, n, k):
    """Operands whose fma chains expose any difference from IEEE fused
    multiply-add with one rounding and gradual underflow."""
    A = inputs.normal(g, (m, k))
    B = inputs.normal(g, (k, n))
    if mode == "subnormal_products":
        A = np.ldexp(A, -70).astype(np.float32); B = np.ldexp(B, -70).astype(np.float32)
    elif mode == "near_min_normal":
        A = np.ldexp(A, -63).astype(np.float32); B = np.ldexp(B, -62).astype(np.float32)
    elif mode == "overflow":
        A = np.ldexp(A, 60).astype(np.float32)
        B = np.ldexp(B, 60 + g.integers(0, 8, B.shape)).astype(np.float32)
    elif mode == "fused_witness":
        a0, a1 = -(1 + 2.0 ** -11), 1 + 2.0 ** -12
        A = np.where(np.arange(k) % 2 == 0, a0, a1)[None, :].repeat(m, 0).astype(np.float32)
        A[1::2] *= -1
        B = np.where(np.arange(k) % 2 == 0, 1.0, a1)[:, None].repeat(n, 1).astype(np.float32)
    elif mode == "subnormal_inputs":
        A = (A.view(np.uint32) & np.uint32(0x807FFFFF)).view(np.float32)
    elif mode == "signed_zeros":
        A = inputs.integers(g, (m, k), -4, 4); B = inputs.integers(g, (k, n), -4, 4)
        A[g.random((m, k)) < 0.2] = -0.0
    elif mode == "ties":
        A = np.ldexp(A, 20).astype(np.float32); B = np.ldexp(B, -20).astype(np.float32)
        A[:, ::3] *= -1
    return np.ascontiguousarray(A, np.float32), np.ascontiguousarray(B, np.float32)


@pytest.mark.parametrize("mode", ["normal", "subnormal_products", "near_min_normal", "overflow",
                                  "fused_witness", "subnormal_inputs", "signed_zeros", "ties"])
@pytest.mark.parametrize("k_block", [64, 0])
def test_matrix_core_chain_equals_fma_chain(rp, mode, k_block):
    """The matrix-core path is allowed only because its single-term updates
    equal the IEEE fma chain: checked here on operands built to expose any
    flush of subnormals, double rounding, wrong zero signs or overflow
    handling, through every launch configuration (matrix-core and vector)."""
    g = inputs.rng(sum(map(ord, mode)) + k_block)
    m, n, k = 96, 80, 256
    A, B = _adversarial(mode, g, m, n, k)
    want = oracle.matmul(A, B, k_block=k_block)
    for name, launch in launches(rp, k_block, True):
        announce("adversarial", mode, k_block, name)
        got = host(rp.matmul(dev(A), dev(B), order=rp.Order(k_block=k_block), launch=launch))
        assert_bits_equal(got, want, f"{mode} {name}")


def _negative_zero_witness(m, n, k):
    """Every output (i, j) has exactly one nonzero product, -2^-160, at
    k = 7 i mod K (row i of A has one nonzero entry there; every row of B
    that some row of A uses is 2^-80): the fused block partial holding it is
    -0, while zero padding past K or the +0 accumulator turns it into +0."""
    A = np.zeros((m, k), np.float32)
    B = np.zeros((k, n), np.float32)
    ks = (7 * np.arange(m)) % k
    A[np.arange(m), ks] = -(2.0 ** -80)
    B[np.unique(ks), :] = 2.0 ** -80
    return A, B


@pytest.mark.parametrize("k", [70, 64, 1, 133])
@pytest.mark.parametrize("k_block", [64, 0])
def test_negative_zero_partials_vanish_in_the_accumulator(rp, k, k_block):
    """A -0 block partial (a negative product below half the smallest subnormal)
    never reaches the output: the accumulator starts at +0, so every output is
    +0 under every launch, with K both a multiple and not a multiple of the
    slice depths, one block (k_block 0) and several."""
    m, n = 70, 66
    A, B = _negative_zero_witness(m, n, k)
    want = oracle.matmul(A, B, k_block=k_block)
    assert not np.signbit(want).any() and not want.any()
    for name, launch in launches(rp, k_block, True):
        announce("negative-zero witness", k, k_block, name)
        got = host(rp.matmul(dev(A), dev(B), order=rp.Order(k_block=k_block), launch=launch))
        assert_bits_equal(got, want, f"K={k} k_block={k_block} {name}")
        got_t = host(rp.matmul(dev(np.ascontiguousarray(A.T)).t(), dev(B),
                               order=rp.Order(k_block=k_block), launch=launch))
        assert_bits_equal(got_t, want, f"transposed A K={k} k_block={k_block} {name}")


GROUP_CASES = [
    # (m, n, k, trans_a, trans_b, bias) per product
    [(300, 260, 512, 1, 0, False), (520, 300, 128, 0, 1, True)],      # one launch, mixed layouts
    [(96, 80, 256, 0, 0, True), (200, 132, 48, 1, 1, False), (64, 64, 1024, 0, 1, False)],
    [(65, 70, 130, 0, 0, True), (33, 17, 64, 1, 0, False)],           # K % 16 != 0: one by one
    [(0, 10, 16, 0, 0, False), (40, 44, 0, 0, 0, True), (70, 72, 96, 0, 0, False)],  # empty ones
]


@pytest.mark.parametrize("case", range(len(GROUP_CASES)))
@pytest.mark.parametrize("k_block,k_inner", [(64, 0), (0, 0), (64, 1)])
def test_matmul_grouped_equals_single_products(rp, case, k_block, k_inner):
    """Every product of a grouped call has the bits of its own matmul call and
    of the oracle -- in one launch (the staged tile) or one by one (other
    shapes and orders)."""
    g = inputs.rng(700 + case * 10 + k_block + k_inner)
    order = rp.Order(k_block=k_block, k_inner=k_inner)
    prods, wants, hosts = [], [], []
    for m, n, k, ta, tb, with_bias in GROUP_CASES[case]:
        A = inputs.normal(g, (k, m) if ta else (m, k))
        B = inputs.normal(g, (n, k) if tb else (k, n))
        bias = inputs.uniform(g, (n,), -0.1, 0.1) if with_bias else None
        wants.append(oracle.matmul(A, B, bias, trans_a=bool(ta), trans_b=bool(tb),
                                   k_block=k_block, k_inner=k_inner))
        dA, dB = dev(A), dev(B)
        prods.append((dA.t() if ta else dA, dB.t() if tb else dB,
                      None if bias is None else dev(bias), None))
    announce("grouped matmul", case, k_block, k_inner)
    outs = rp.matmul_grouped(prods, order=order)
    for i, (out, want, p) in enumerate(zip(outs, wants, prods)):
        assert_bits_equal(host(out), want, f"product {i} vs oracle")
        single = rp.matmul(p[0], p[1], p[2], order=order)
        assert same_bits(out, single), f"product {i} vs its own matmul"


def test_matmul_grouped_training_step_shapes(rp):
    """The feed-forward training step's gradient pairs at full size (weight
    gradient, K = 4096 tokens, and input gradient), grouped, against their own
    matmul calls on every output and the oracle on samples."""
    g = inputs.rng(777)
    G = inputs.normal(g, (4096, 3072), var=0.1)
    dH = inputs.normal(g, (4096, 768), var=1e-4)
    W2 = inputs.normal(g, (3072, 768), var=4e-4)
    dG, dW, W = dev(G), dev(dH), dev(W2)
    announce("grouped matmul dW2 + dG")
    gw, gg = rp.matmul_grouped([(dG.t(), dW, None, None), (dW, W.t(), None, None)])
    assert same_bits(gw, rp.matmul(dG.t(), dW)) and same_bits(gg, rp.matmul(dW, W.t()))
    r, c = inputs.sample_indices(8, 512, 3072, 768)
    assert_bits_equal(host(gw)[r, c], oracle.matmul_at(G, dH, r, c, trans_a=True), "dW2")
    r, c = inputs.sample_indices(9, 512, 4096, 3072)
    assert_bits_equal(host(gg)[r, c], oracle.matmul_at(dH, W2, r, c, trans_b=True), "dG")


CAUSAL_SHAPES = [(1, 2, 300, 300, 64), (2, 3, 257, 257, 100), (1, 1, 1024, 1024, 128),
                 (2, 2, 200, 130, 200)]


@pytest.mark.parametrize("shape", CAUSAL_SHAPES)
@pytest.mark.parametrize("k_block,k_inner", [(64, 0), (0, 0), (32, 1)])
def test_bmm_causal_output_lower_triangle(rp, shape, k_block, k_inner):
    """REPOPS_CAUSAL_OUTPUT: every output with j <= i has repops_bmm's bits
    (and the oracle's) under every launch; the rest is unspecified."""
    b0, b1, m, n, k = shape
    g = inputs.rng(900 + m + k + k_block)
    A = inputs.normal(g, (b0, b1, m, k))
    B = inputs.normal(g, (b0, b1, n, k))
    want = oracle.bmm(A, B, alpha=0.125, trans_b=True, k_block=k_block, k_inner=k_inner)
    lower = np.tril(np.ones((m, n), bool))
    order = rp.Order(k_block=k_block, k_inner=k_inner)
    import torch
    for name, launch in [("auto", None)] + launches(rp, k_block, k_inner == 0):
        announce("bmm causal output", shape, k_block, k_inner, name)
        C = torch.full((b0, b1, m, n), float("nan"), device="cuda:0")
        rp.bmm_raw(b0, b1, m, n, k, dev(A), b1 * m * k, m * k, k, 0, dev(B), b1 * n * k, n * k, k,
                   1, 0.125, C, b1 * m * n, m * n, n, order=order, launch=launch,
                   causal=rp.CAUSAL_OUTPUT)
        got = host(C)
        assert_bits_equal(np.where(lower, got, 0), np.where(lower, want, 0), f"{shape} {name}")


@pytest.mark.parametrize("shape", CAUSAL_SHAPES)
@pytest.mark.parametrize("k_block,k_inner", [(64, 0), (0, 0), (32, 1), (128, 0)])
def test_bmm_causal_a_is_bitwise_bmm(rp, shape, k_block, k_inner):
    """REPOPS_CAUSAL_A with A zero above its diagonal (as a causal softmax
    leaves P, signed zeros included): every output equals repops_bmm and the
    oracle bit for bit under every launch -- the skipped k blocks held only
    zero products."""
    b0, b1, m, n, k = shape
    k = m  # P is square per batch element
    g = inputs.rng(950 + m + k_block)
    A = inputs.normal(g, (b0, b1, m, k))
    upper = np.triu(np.ones((m, k), bool), 1)
    A[..., upper] = 0.0
    A[..., :, k - 1][..., :m - 1] = -0.0   # negative zeros above the diagonal too
    A = np.ascontiguousarray(A, np.float32)
    B = inputs.normal(g, (b0, b1, k, n))
    want = oracle.bmm(A, B, k_block=k_block, k_inner=k_inner)
    order = rp.Order(k_block=k_block, k_inner=k_inner)
    import torch
    for name, launch in [("auto", None)] + launches(rp, k_block, k_inner == 0):
        announce("bmm causal A", shape, k_block, k_inner, name)
        C = torch.empty((b0, b1, m, n), device="cuda:0")
        rp.bmm_raw(b0, b1, m, n, k, dev(A), b1 * m * k, m * k, k, 0, dev(B), b1 * k * n, k * n, n,
                   0, 1.0, C, b1 * m * n, m * n, n, order=order, launch=launch,
                   causal=rp.CAUSAL_A)
        assert_bits_equal(host(C), want, f"{shape} {name}")

"""GPU parity on the five workloads at full size (0 ULP).

Where the oracle can take every output in seconds it does; at the large
shapes it computes sampled outputs one by one (each from the original seeded
inputs, never from a GPU result), and the launch configurations are compared
with each other on every output.  Composite programs are checked end to end
on rows (MLP) or on whole heads (attention) that the oracle recomputes from
the original inputs.
"""
import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal
from gpu_util import announce, dev, host, same_bits
from paper_2502_19405_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2502_19405_amd import repops
    repops.load()
    return repops


def gemm_launches(rp, include_simple=True):
    out = [("simple", rp.Launch(rp.LAUNCH_GEMM_SIMPLE))] if include_simple else []
    out += [(f"tiled{i}:{n}", rp.Launch(rp.LAUNCH_GEMM_TILED, (i,)))
            for i, n in enumerate(rp.gemm_configs(rp.LAUNCH_GEMM_TILED))]
    out += [(f"mfma{i}:{n}", rp.Launch(rp.LAUNCH_GEMM_MFMA, (i,)))
            for i, n in enumerate(rp.gemm_configs(rp.LAUNCH_GEMM_MFMA))]
    return out


# ---------------------------------------------------------------- 256^3 + softmax

def test_gemm256_softmax256_full(rp):
    d = inputs.gemm256_softmax256()
    want = oracle.matmul(d["A"], d["B"])
    for name, launch in gemm_launches(rp):
        announce("gemm256", name)
        assert_bits_equal(host(rp.matmul(dev(d["A"]), dev(d["B"]), launch=launch)), want, name)
    want_s = oracle.softmax_rows(d["S"])
    for name, launch in [("auto", None), ("generic", rp.Launch(rp.LAUNCH_ROWS_GENERIC))] + [
            (f"wave{w}", rp.Launch(rp.LAUNCH_ROWS_WAVE, (w,))) for w in (1, 2, 4, 8)]:
        announce("softmax256", name)
        assert_bits_equal(host(rp.softmax_rows(dev(d["S"]), launch=launch)), want_s, name)


# ---------------------------------------------------------------- 2048^3 + bias

def test_gemm2048_bias_sampled_and_cross_launch(rp):
    d = inputs.gemm2048_bias()
    rows, cols = inputs.sample_indices(1, 4096, 2048, 2048)
    want = oracle.matmul_at(d["A"], d["B"], rows, cols, bias=d["bias"])
    dA, dB, dbias = dev(d["A"]), dev(d["B"]), dev(d["bias"])
    ref = None
    for name, launch in gemm_launches(rp):
        announce("gemm2048", name)
        C = rp.matmul(dA, dB, dbias, launch=launch)
        assert_bits_equal(host(C)[rows, cols], want, name)
        if ref is None:
            ref = C
        else:
            assert same_bits(C, ref), f"{name} differs from the first launch configuration"


def test_gemm2048_integer_exact(rp):
    d = inputs.gemm2048_int()
    exact = d["A"].astype(np.float64) @ d["B"].astype(np.float64)
    for name, launch in gemm_launches(rp, include_simple=False):
        announce("gemm2048 int", name)
        got = host(rp.matmul(dev(d["A"]), dev(d["B"]), dev(d["bias"]), launch=launch))
        assert np.array_equal(got, (exact + d["bias"]).astype(np.float32)), name
        got0 = host(rp.matmul(dev(d["A"]), dev(d["B"]), launch=launch))
        assert np.array_equal(got0, exact.astype(np.float32)), name


# ---------------------------------------------------------------- DistilBERT MLP

def test_distilbert_mlp_rows_end_to_end(rp):
    from paper_2502_19405_amd import pipelines
    d = inputs.distilbert_mlp()
    announce("mlp pipeline")
    out = pipelines.mlp_forward(dev(d["X"]), dev(d["W1"]), dev(d["b1"]), dev(d["W2"]),
                                dev(d["b2"]), dev(d["gamma"]), dev(d["beta"]), keep=True)
    rows = np.array([0, 1, 63, 64, 1000, 2047, 2048, 3333, 4094, 4095])
    X = np.ascontiguousarray(d["X"][rows])
    H1 = oracle.matmul(X, d["W1"], d["b1"])
    G = oracle.gelu(H1)
    H2 = oracle.matmul(G, d["W2"], d["b2"])
    Y = oracle.layernorm_rows(H2, d["gamma"], d["beta"], eps=1e-5)
    for key, want in (("H1", H1), ("G", G), ("H2", H2), ("Y", Y)):
        assert_bits_equal(host(out[key])[rows], want, key)


def test_distilbert_shaped_gelu_and_layernorm_full(rp):
    g = inputs.rng(33)
    H = inputs.normal(g, (4096, 3072), var=0.31)
    announce("gelu 4096x3072")
    assert_bits_equal(host(rp.gelu(dev(H))), oracle.gelu(H), "gelu")
    d = inputs.distilbert_mlp()
    Z = inputs.normal(g, (4096, 768), var=0.5)
    want = oracle.layernorm_rows(Z, d["gamma"], d["beta"], eps=1e-5)
    for launch in (None, rp.Launch(rp.LAUNCH_ROWS_GENERIC), rp.Launch(rp.LAUNCH_ROWS_WAVE, (8,))):
        announce("layernorm 4096x768", launch)
        got = rp.layernorm_rows(dev(Z), dev(d["gamma"]), dev(d["beta"]), eps=1e-5, launch=launch)
        assert_bits_equal(host(got), want, str(launch))


# ---------------------------------------------------------------- Llama attention

def test_llama_attention_heads_end_to_end(rp):
    from paper_2502_19405_amd import pipelines
    d = inputs.llama_attention()
    B, T, D, H = 4, 1024, 4096, 32
    hd = D // H
    announce("attention pipeline")
    out = pipelines.attention_forward(dev(d["X"]), dev(d["Wq"]), dev(d["Wk"]), dev(d["Wv"]),
                                      dev(d["Wo"]), B, T, H, keep=True)
    S, P, O = host(out["S"]), host(out["P"]), host(out["O"])
    alpha = np.float32(pipelines.attention_scale(hd))
    for b, h in ((0, 0), (3, 31)):
        announce("attention oracle head", b, h)
        Xb = np.ascontiguousarray(d["X"][b * T:(b + 1) * T])
        cols = slice(h * hd, (h + 1) * hd)
        Qh = oracle.matmul(Xb, np.ascontiguousarray(d["Wq"][:, cols]))
        Kh = oracle.matmul(Xb, np.ascontiguousarray(d["Wk"][:, cols]))
        Vh = oracle.matmul(Xb, np.ascontiguousarray(d["Wv"][:, cols]))
        Sh = oracle.bmm(Qh[None, None], np.ascontiguousarray(Kh)[None, None], alpha=alpha,
                        trans_b=True)[0, 0]
        Ph = oracle.softmax_rows(Sh, causal_period=T)
        Oh = oracle.matmul(Ph, Vh)
        assert_bits_equal(S[b, h], Sh, f"S[{b},{h}]")
        assert_bits_equal(P.reshape(B, H, T, T)[b, h], Ph, f"P[{b},{h}]")
        assert_bits_equal(O[b * T:(b + 1) * T, cols], Oh, f"O[{b},{h}]")


def test_llama_attention_projection_gemms_sampled(rp):
    d = inputs.llama_attention()
    rows, cols = inputs.sample_indices(4, 1024, 4096, 4096)
    dX = dev(d["X"])
    for w in ("Wq", "Wo"):
        want = oracle.matmul_at(d["X"], d[w], rows, cols)
        for name, launch in gemm_launches(rp, include_simple=False):
            announce("projection", w, name)
            got = host(rp.matmul(dX, dev(d[w]), launch=launch))
            assert_bits_equal(got[rows, cols], want, f"{w} {name}")


def test_llama_attention_score_bmm_and_softmax_full_shape(rp):
    """QK^T and PV at their full shapes (4 x 32 heads) on seeded operands of
    the projections' distribution, sampled; causal softmax over all 131072 rows
    of 1024, every output."""
    g = inputs.rng(44)
    B, T, D, H = 4, 1024, 4096, 32
    hd = D // H
    Q = inputs.normal(g, (B * T, D), var=1.64)
    K = inputs.normal(g, (B * T, D), var=1.64)
    alpha = np.float32(1 / np.sqrt(128.0))
    b0, b1, r, c = inputs.sample_indices(5, 2048, B, H, T, T)
    want = oracle.bmm_at_raw(B, H, T, T, hd, Q.ravel(), T * D, hd, D, 0, K.ravel(), T * D, hd, D, 1,
                             alpha, b0, b1, r, c)
    import torch
    S = torch.empty((B, H, T, T), device="cuda:0")
    for name, launch in gemm_launches(rp, include_simple=False):
        announce("QK^T bmm", name)
        rp.bmm_raw(B, H, T, T, hd, dev(Q), T * D, hd, D, 0, dev(K), T * D, hd, D, 1, float(alpha),
                   S, H * T * T, T * T, T, launch=launch)
        assert_bits_equal(host(S)[b0, b1, r, c], want, name)
    Sx = inputs.normal(g, (B * H * T, T), var=4.0)
    want_p = oracle.softmax_rows(Sx, causal_period=T)
    dS = dev(Sx)
    for launch in (None, rp.Launch(rp.LAUNCH_ROWS_WAVE, (1,)), rp.Launch(rp.LAUNCH_ROWS_GENERIC)):
        announce("causal softmax 131072x1024", launch)
        assert_bits_equal(host(rp.softmax_rows(dS, causal_period=T, launch=launch)), want_p,
                          str(launch))


# ---------------------------------------------------------------- Llama backward

@pytest.fixture(scope="module")
def backward_data():
    return inputs.llama_linear_backward()


def test_llama_linear_backward_sampled_across_tiles(rp, backward_data):
    from paper_2502_19405_amd import pipelines
    d = backward_data
    r1, c1 = inputs.sample_indices(6, 1024, 8192, 4096)
    r2, c2 = inputs.sample_indices(7, 1024, 4096, 14336)
    want_dx = oracle.matmul_at(d["dY"], d["W"], r1, c1, trans_b=True)
    want_dw = oracle.matmul_at(d["X"], d["dY"], r2, c2, trans_a=True)
    dX_, dY_, W_ = dev(d["X"]), dev(d["dY"]), dev(d["W"])
    ref = None
    for name, launch in gemm_launches(rp, include_simple=False):
        announce("linear backward", name)
        gx, gw = pipelines.linear_backward(dX_, dY_, W_, gemm_launch=launch)
        assert_bits_equal(host(gx)[r1, c1], want_dx, f"dX {name}")
        assert_bits_equal(host(gw)[r2, c2], want_dw, f"dW {name}")
        if ref is None:
            ref = (gx, gw)
        else:
            assert same_bits(gx, ref[0]) and same_bits(gw, ref[1]), name

"""GPU parity on the five workloads at full size (0 ULP).

Every output of every workload is checked against the oracle: where the oracle
takes them all in seconds (the 256^3 and 2048^3 GEMMs, the feed-forward block)
it runs in the test; at the large shapes (the attention block, the linear
layer's backward products, the feed-forward training step at 4096 tokens) the
test compares SHA-256 digests of whole outputs with digests of the oracle's
outputs stored by tests/golden/make_oracle_digests.py, and computes sampled
outputs with the oracle one by one so that a mismatch is named.  Each workload
runs under at least three launch configurations (matrix-core table entries and
vector-FMA tiles): the first launch's outputs against the oracle, every other
launch's outputs against the first one's on every element.
"""
import numpy as np
import pytest

import digests
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

def test_gemm2048_bias_full_every_launch(rp):
    d = inputs.gemm2048_bias()
    announce("gemm2048 oracle (every output)")
    want = oracle.matmul(d["A"], d["B"], d["bias"])
    dA, dB, dbias = dev(d["A"]), dev(d["B"]), dev(d["bias"])
    for name, launch in gemm_launches(rp):
        announce("gemm2048", name)
        assert_bits_equal(host(rp.matmul(dA, dB, dbias, launch=launch)), want, name)


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

def mlp_launches(rp):
    """Matrix-core entries 0 (staged 128x128), 2 (register-staged), 5 (64x64),
    7 (staged 256x128) and 9 (the persistent ring form, which the first product's
    768 tiles take), and both vector-FMA tiles."""
    return [(n, l) for n, l in gemm_launches(rp, include_simple=False)
            if n.split(":")[0] in ("mfma0", "mfma2", "mfma5", "mfma7", "mfma9", "tiled0",
                                   "tiled1")]


def test_distilbert_mlp_block_full_every_launch(rp):
    from paper_2502_19405_amd import pipelines
    from oracle import compose
    d = inputs.distilbert_mlp()
    announce("mlp oracle (every output)")
    want = compose.mlp_forward(d["X"], d["W1"], d["b1"], d["W2"], d["b2"], d["gamma"], d["beta"])
    args = [dev(d[k]) for k in ("X", "W1", "b1", "W2", "b2", "gamma", "beta")]
    for name, launch in mlp_launches(rp):
        announce("mlp pipeline", name)
        out = pipelines.mlp_forward(*args, gemm_launch=launch, keep=True)
        for key in ("H1", "G", "H2", "Y"):
            assert_bits_equal(host(out[key]), want[key], f"{key} {name}")


def test_distilbert_mlp_training_step_4096_tokens_every_launch(rp):
    """Two whole training steps of the feed-forward block at 4096 tokens --
    forward, every gradient (the dW products contract over the 4096 tokens,
    the dX products over 3072 and 768 features), AdamW of all parameters --
    equal the oracle's composition on every output (stored digests), with the
    automatic launches (gradient products grouped) and under four GEMM launch
    configurations."""
    import torch
    from paper_2502_19405_amd import pipelines
    from oracle.compose import MLP_PARAM_NAMES
    tokens = 4096
    d = inputs.distilbert_mlp(tokens=tokens)
    dYs = digests.train_step_gradients(tokens)
    ins = dict(d)
    ins.update({f"dY_step{i}": v for i, v in enumerate(dYs, start=1)})
    want = digests.entry("mlp_train_step_4096", ins)
    Xd = dev(d["X"])
    ref = None
    for name, launch in [("auto (grouped gradient products)", None)] + [
            (n, l) for n, l in mlp_launches(rp)
            if n.split(":")[0] in ("mfma0", "mfma5", "mfma7", "tiled1")]:
        st = pipelines.MlpTrainState(*(dev(d[k]) for k in MLP_PARAM_NAMES))
        outs = {}
        for step, dY in enumerate(dYs, start=1):
            announce("mlp train step 4096", name, step)
            Yg, dXg = pipelines.mlp_train_step(st, Xd, dev(dY), gemm_launch=launch)
            torch.cuda.synchronize()
            outs[f"step{step}/Y"] = Yg.clone()
            outs[f"step{step}/dX"] = dXg.clone()
            for pn, gg, pg in zip(MLP_PARAM_NAMES, st.g, st.p):
                outs[f"step{step}/grad_{pn}"] = gg.clone()
                outs[f"step{step}/param_{pn}"] = pg.clone()
            outs[f"step{step}/exp_avg"] = st.exp_avg.clone()
            outs[f"step{step}/exp_avg_sq"] = st.exp_avg_sq.clone()
        if ref is None:
            for key, t in outs.items():
                assert digests.sha256_of(host(t)) == want[key], f"{key} {name} differs from the oracle"
            ref = outs
        else:
            for key, t in outs.items():
                assert same_bits(t, ref[key]), f"{key} {name} differs from the first launch"


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
        low = np.tril(np.ones((T, T), bool))  # the causal product's defined part
        assert_bits_equal(np.where(low, S[b, h], 0), np.where(low, Sh, 0), f"S[{b},{h}]")
        assert_bits_equal(P.reshape(B, H, T, T)[b, h], Ph, f"P[{b},{h}]")
        assert_bits_equal(O[b * T:(b + 1) * T, cols], Oh, f"O[{b},{h}]")


def test_llama_attention_block_full_every_launch(rp):
    """The whole attention block (Q, K, V projections, QK^T, causal softmax,
    PV, output projection) at its full shape: every intermediate and the
    output equal the oracle's composition (stored digests) under the first
    launch configuration and equal that launch's bits under every other
    matrix-core and vector-FMA launch; sampled projection outputs are also
    recomputed by the oracle one by one."""
    from paper_2502_19405_amd import pipelines
    d = inputs.llama_attention()
    want = digests.entry("llama_attention", d)
    args = [dev(d[k]) for k in ("X", "Wq", "Wk", "Wv", "Wo")]
    rows, cols = inputs.sample_indices(4, 512, 4096, 4096)
    samples = {"Q": oracle.matmul_at(d["X"], d["Wq"], rows, cols)}
    ref = None
    for name, launch in [("auto (grouped projections)", None)] + gemm_launches(
            rp, include_simple=False):
        announce("attention block", name)
        out = pipelines.attention_forward(*args, 4, 1024, 32, gemm_launch=launch, keep=True)
        assert_bits_equal(host(out["Q"])[rows, cols], samples["Q"], f"Q samples {name}")
        # the causal score product leaves S above each head's diagonal unspecified
        import torch
        lower = torch.tril(torch.ones((1024, 1024), dtype=torch.bool, device="cuda:0"))
        out["S"] = torch.where(lower, out["S"], torch.zeros((), device="cuda:0"))
        if ref is None:
            for key in ("Q", "K", "V", "S", "P", "O", "out"):
                dk = "S_lower" if key == "S" else key
                assert digests.sha256_of(host(out[key])) == want[dk], (
                    f"{key} {name} differs from the oracle")
            ref = out
        else:
            for key in ("Q", "K", "V", "S", "P", "O", "out"):
                assert same_bits(out[key], ref[key]), f"{key} {name} differs from the first launch"
        del out


def test_llama_attention_score_bmm_and_softmax_full_shape(rp):
    """QK^T and PV at their full shapes (4 x 32 heads) on seeded operands of
    the projections' distribution, sampled outputs against the oracle under
    every matrix-core and vector-FMA launch; causal softmax over all 131072
    rows of 1024, every output."""
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
    # PV: the causal probabilities times V's head columns, written in place
    # into O's head columns
    V = inputs.normal(g, (B * T, D), var=1.64)
    b0, b1, r, c = inputs.sample_indices(6, 2048, B, H, T, hd)
    want_o = oracle.bmm_at_raw(B, H, T, hd, T, want_p.ravel(), H * T * T, T * T, T, 0,
                               V.ravel(), T * D, hd, D, 0, 1.0, b0, b1, r, c)
    dP, dV = dev(want_p), dev(V)
    O = torch.empty((B * T, D), device="cuda:0")
    for name, launch in gemm_launches(rp, include_simple=False):
        announce("PV bmm", name)
        rp.bmm_raw(B, H, T, hd, T, dP, H * T * T, T * T, T, 0, dV, T * D, hd, D, 0, 1.0,
                   O, T * D, hd, D, launch=launch)
        Oh = host(O).reshape(B, T, H, hd)
        assert_bits_equal(Oh[b0, r, b1, c], want_o, name)


# ---------------------------------------------------------------- Llama backward

@pytest.fixture(scope="module")
def backward_data():
    return inputs.llama_linear_backward()


def test_llama_linear_backward_full_every_launch(rp, backward_data):
    """dX = dY W^T (K = 14336) and dW = X^T dY (K = 8192 tokens) at full size:
    every output equals the oracle's (stored digests) under the first launch
    and that launch's bits under every other matrix-core and vector-FMA
    launch; sampled outputs are recomputed by the oracle one by one."""
    from paper_2502_19405_amd import pipelines
    d = backward_data
    want = digests.entry("llama_linear_backward", d)
    r1, c1 = inputs.sample_indices(6, 512, 8192, 4096)
    r2, c2 = inputs.sample_indices(7, 512, 4096, 14336)
    want_dx = oracle.matmul_at(d["dY"], d["W"], r1, c1, trans_b=True)
    want_dw = oracle.matmul_at(d["X"], d["dY"], r2, c2, trans_a=True)
    dX_, dY_, W_ = dev(d["X"]), dev(d["dY"]), dev(d["W"])
    ref = None
    for name, launch in [("auto (grouped)", None)] + gemm_launches(rp, include_simple=False):
        announce("linear backward", name)
        gx, gw = pipelines.linear_backward(dX_, dY_, W_, gemm_launch=launch)
        assert_bits_equal(host(gx)[r1, c1], want_dx, f"dX samples {name}")
        assert_bits_equal(host(gw)[r2, c2], want_dw, f"dW samples {name}")
        if ref is None:
            assert digests.sha256_of(host(gx)) == want["dX"], f"dX {name} differs from the oracle"
            assert digests.sha256_of(host(gw)) == want["dW"], f"dW {name} differs from the oracle"
            ref = (gx, gw)
        else:
            assert same_bits(gx, ref[0]), f"dX {name} differs from the first launch"
            assert same_bits(gw, ref[1]), f"dW {name} differs from the first launch"

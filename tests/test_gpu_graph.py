"""Library calls captured in one HIP graph: every replay gives the bits of the
eager calls and of the CPU oracle (the library allocates and clears nothing,
so its launches capture as they run).  Between replays the outputs are
cleared by eager fill kernels and the host synchronizes, so each replay is
checked on its own."""
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


def test_graph_replays_match_eager_and_oracle(rp):
    import torch
    g = inputs.rng(901)
    Xh = inputs.normal(g, (512, 768))
    gamh = 1 + inputs.uniform(g, (768,), -0.1, 0.1)
    beth = inputs.uniform(g, (768,), -0.1, 0.1)
    Sh = inputs.normal(g, (96, 4096), var=4.0)
    Ah = inputs.normal(g, (256, 256))
    Bh = inputs.normal(g, (256, 256))
    Rh = inputs.normal(g, (64, 8192))
    X, gam, bet, S, A, B, R = (dev(a) for a in (Xh, gamh, beth, Sh, Ah, Bh, Rh))
    Y, P, Q = torch.empty_like(X), torch.empty_like(S), torch.empty_like(R)
    C = torch.empty(256, 256, device="cuda:0")

    def calls():
        rp.layernorm_rows(X, gam, bet, out=Y)
        rp.softmax_rows(S, causal_period=1000, out=P)  # split rows with a mask
        rp.matmul(A, B, out=C)
        rp.rmsnorm_rows(R, out=Q)

    announce("graph", "eager")
    calls()
    torch.cuda.synchronize()
    eager = [host(t).copy() for t in (Y, P, C, Q)]
    want = [oracle.layernorm_rows(Xh, gamh, beth, eps=1e-5),
            oracle.softmax_rows(Sh, causal_period=1000),
            oracle.matmul(Ah, Bh),
            oracle.rmsnorm_rows(Rh, None, eps=1e-5)]
    for got, w, name in zip(eager, want, ("layernorm", "softmax", "matmul", "rmsnorm")):
        assert_bits_equal(got, w, f"eager {name}")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        calls()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        calls()
    for rep in range(3):
        announce("graph", "replay", rep)
        for t in (Y, P, C, Q):
            t.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for t, e, name in zip((Y, P, C, Q), eager, ("layernorm", "softmax", "matmul", "rmsnorm")):
            assert_bits_equal(host(t), e, f"replay {rep} {name}")


def test_graph_model_blocks_match_eager_and_oracle(rp):
    # The model-shaped compositions captured whole: the feed-forward block (product
    # with the GELU epilogue, product, LayerNorm) and the attention block (grouped
    # projections, causal score product, causal softmax, causal value product,
    # output projection).  Every replay gives the eager bits; eager gives the
    # oracle compositions' bits.
    import torch

    from oracle import compose
    from paper_2502_19405_amd import pipelines
    g = inputs.rng(902)
    t, h, f = 192, 64, 256
    mh = {"X": inputs.normal(g, (t, h)), "W1": inputs.normal(g, (h, f), var=1.0 / h),
          "b1": inputs.uniform(g, (f,), -0.1, 0.1), "W2": inputs.normal(g, (f, h), var=1.0 / f),
          "b2": inputs.uniform(g, (h,), -0.1, 0.1), "gamma": 1 + inputs.uniform(g, (h,), -0.1, 0.1),
          "beta": inputs.uniform(g, (h,), -0.1, 0.1)}
    batch, seq, heads, d = 2, 128, 4, 128
    ah = {"X": inputs.normal(g, (batch * seq, d))}
    for w in ("Wq", "Wk", "Wv", "Wo"):
        ah[w] = inputs.normal(g, (d, d), var=1.0 / d)
    m = {k: dev(v) for k, v in mh.items()}
    a = {k: dev(v) for k, v in ah.items()}
    margs = (m["X"], m["W1"], m["b1"], m["W2"], m["b2"], m["gamma"], m["beta"])
    aargs = (a["X"], a["Wq"], a["Wk"], a["Wv"], a["Wo"], batch, seq, heads)

    def calls():
        return (pipelines.mlp_forward(*margs, keep=True),
                pipelines.attention_forward(*aargs, keep=True))

    announce("graph blocks", "eager")
    mo, ao = calls()
    torch.cuda.synchronize()
    want_m = compose.mlp_forward(mh["X"], mh["W1"], mh["b1"], mh["W2"], mh["b2"], mh["gamma"],
                                 mh["beta"])
    want_a = compose.attention_forward(ah["X"], ah["Wq"], ah["Wk"], ah["Wv"], ah["Wo"], batch,
                                       seq, heads)
    lower = torch.tril(torch.ones(seq, seq, dtype=torch.bool, device="cuda:0"))

    def results(mo, ao):
        r = {f"mlp {k}": host(mo[k]).copy() for k in ("H1", "G", "H2", "Y")}
        r.update({f"attn {k}": host(ao[k]).copy() for k in ("Q", "K", "V", "P", "O", "out")})
        # the score product is specified at and below each head's diagonal only
        r["attn S lower"] = host(torch.where(lower, ao["S"], torch.zeros_like(ao["S"]))).copy()
        return r
    eager = results(mo, ao)
    for k in ("H1", "G", "H2", "Y"):
        assert_bits_equal(eager[f"mlp {k}"], want_m[k], f"eager mlp {k}")
    for k in ("Q", "K", "V", "P", "O", "out"):
        assert_bits_equal(eager[f"attn {k}"], want_a[k], f"eager attention {k}")
    import numpy as np
    S_lower = np.where(np.tril(np.ones((seq, seq), bool)), want_a["S"], np.float32(0))
    assert_bits_equal(eager["attn S lower"], S_lower.astype(np.float32), "eager attention S")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        calls()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        gm, ga = calls()
    for rep in range(3):
        announce("graph blocks", "replay", rep)
        for t_ in list(gm.values()) + list(ga.values()):
            t_.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = results(gm, ga)
        for k, e in eager.items():
            assert_bits_equal(got[k], e, f"replay {rep} {k}")

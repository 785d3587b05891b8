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

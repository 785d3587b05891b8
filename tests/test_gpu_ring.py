"""GPU parity of the persistent ring form of the default matrix-core tile
(table entry 9) against the CPU oracle, 0 ULP.

The ring form runs only where every tile makes whole ring turns (K a multiple
of 64 with the default 64-deep blocks) and there are more 128 x 128 tiles than
compute units, so these shapes have a few hundred tiles: each workgroup then
takes several tiles in turn, and the last ring turn of each tile loads the next
tile's first slices.  Covered: an odd and an even number of ring turns per
tile, ragged row and column edges, every transposition, bias, the GELU and
GELU-backward epilogues, batched products, the lower-triangle score product
of causal attention, and replays of both score products captured in a HIP
graph.  Shapes the ring form declines (K not a multiple
of 64, other block lengths, few tiles) run entry 0's kernels and are covered by
the other GEMM tests, which run every table entry.
"""
import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal
from gpu_util import announce, dev, host
from paper_2502_19405_amd import inputs

pytestmark = pytest.mark.gpu

RING = 9


@pytest.fixture(scope="module")
def rp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2502_19405_amd import repops
    repops.load()
    assert repops.gemm_configs(repops.LAUNCH_GEMM_MFMA)[RING].endswith("/ring")
    return repops


def ring_launch(rp):
    return rp.Launch(rp.LAUNCH_GEMM_MFMA, (RING,))


# (m, n, k): 306 tiles with ragged edges and one ring turn per tile; 288 tiles,
# three turns (an odd count: the last turn uses the first partial set); 300
# tiles, four turns
SHAPES = [(2100, 2200, 64), (2048, 2304, 192), (1920, 2560, 256)]


@pytest.mark.parametrize("shape", SHAPES)
def test_ring_matmul_every_transposition(rp, shape):
    m, n, k = shape
    g = inputs.rng(9100 + m + k)
    A = inputs.normal(g, (m, k))
    B = inputs.normal(g, (k, n))
    bias = inputs.uniform(g, (n,), -0.1, 0.1)
    want = oracle.matmul(A, B, bias)
    dA, dB, dbias = dev(A), dev(B), dev(bias)
    dAt, dBt = dev(np.ascontiguousarray(A.T)), dev(np.ascontiguousarray(B.T))
    for ta in (0, 1):
        for tb in (0, 1):
            announce("ring matmul", shape, ta, tb)
            a = dAt.t() if ta else dA
            b = dBt.t() if tb else dB
            got = rp.matmul(a, b, dbias, launch=ring_launch(rp))
            assert_bits_equal(host(got), want, f"ring {shape} trans {ta}{tb}")


def test_ring_gelu_epilogues(rp):
    m, n, k = 2100, 2200, 128
    g = inputs.rng(9200)
    A = (inputs.normal(g, (m, k)) * np.float32(1.5 / np.sqrt(k))).astype(np.float32)
    B = inputs.normal(g, (k, n))
    bias = inputs.uniform(g, (n,), -2.0, 2.0)
    X = inputs.uniform(g, (m, n), -4.0, 4.0)
    H = oracle.matmul(A, B, bias)
    announce("ring matmul_gelu")
    h, gl = rp.matmul_gelu(dev(A), dev(B), dev(bias), launch=ring_launch(rp))
    assert_bits_equal(host(h), H, "ring H")
    assert_bits_equal(host(gl), oracle.gelu(H), "ring G")
    announce("ring matmul_gelu_backward")
    got = rp.matmul_gelu_backward(dev(A), dev(B), dev(X), launch=ring_launch(rp))
    assert_bits_equal(host(got), oracle.gelu_backward(X, oracle.matmul(A, B)), "ring dG")


def test_ring_bmm_dense_and_causal_scores(rp):
    # 4 x 8 batch elements of 512 x 512 outputs (16 tiles each, 512 in all),
    # alpha in the epilogue; then the lower-triangle score product (10 tiles per
    # element, 320 in all), compared at and below each element's diagonal
    b0, b1, s, k = 4, 8, 512, 128
    g = inputs.rng(9300)
    Q = inputs.normal(g, (b0, b1, s, k))
    K = inputs.normal(g, (b0, b1, s, k))
    alpha = np.float32(1.0 / np.sqrt(k))
    want = oracle.bmm(Q, K, alpha=float(alpha), trans_b=True)
    dQ = dev(Q)
    dKt = dev(K).transpose(2, 3)
    announce("ring bmm dense")
    got = rp.bmm(dQ, dKt, alpha=float(alpha), launch=ring_launch(rp))
    assert_bits_equal(host(got), want, "ring bmm")
    import torch
    S = torch.full((b0, b1, s, s), float("nan"), device="cuda:0")
    announce("ring bmm causal scores")
    rp.bmm_raw(b0, b1, s, s, k, dQ, b1 * s * k, s * k, k, 0, dev(K), b1 * s * k, s * k, k, 1,
               float(alpha), S, b1 * s * s, s * s, s, launch=ring_launch(rp),
               causal=rp.CAUSAL_OUTPUT)
    lower = np.tril(np.ones((s, s), bool))
    got = host(S)
    assert_bits_equal(np.where(lower, got, np.float32(0)), np.where(lower, want, np.float32(0)),
                      "ring causal scores")


def test_ring_equals_entry0_on_the_feed_forward_shapes(rp):
    # the feed-forward products at 4096 tokens under the ring form and entry 0:
    # the same bits (the oracle pins entry 0 on these shapes in the workload
    # tests).  X W1 and dH2 W2^T have 768 tiles and run the ring form; G W2 (192
    # tiles) and G^T X (144) have fewer tiles than compute units and run entry
    # 0's kernel under either launch.
    import torch
    g = inputs.rng(9400)
    X = dev(inputs.normal(g, (4096, 768)))
    W1 = dev(inputs.normal(g, (768, 3072), var=1.0 / 768))
    G = dev(inputs.normal(g, (4096, 3072)))
    W2 = dev(inputs.normal(g, (3072, 768), var=1.0 / 3072))
    dH2 = dev(inputs.normal(g, (4096, 768)))
    for name, a, b in (("X W1", X, W1), ("dH2 W2^T", dH2, W2.t()), ("G W2", G, W2),
                       ("G^T X", G.t(), X)):
        announce("ring vs entry 0", name)
        r = rp.matmul(a, b, launch=ring_launch(rp))
        e = rp.matmul(a, b, launch=rp.Launch(rp.LAUNCH_GEMM_MFMA, (0,)))
        assert torch.equal(r.view(torch.int32), e.view(torch.int32)), name


def test_ring_under_graph_replay(rp):
    # The dense and lower-triangle score products of the bmm test above in the
    # ring form, captured in one HIP graph: every replay (with eager work and a
    # synchronisation between replays) gives the eager bits, and those are
    # the oracle's.
    import torch
    b0, b1, s, k = 4, 8, 512, 128
    g = inputs.rng(9500)
    Q = inputs.normal(g, (b0, b1, s, k))
    K = inputs.normal(g, (b0, b1, s, k))
    alpha = float(np.float32(1.0 / np.sqrt(k)))
    want = oracle.bmm(Q, K, alpha=alpha, trans_b=True)
    dQ, dK = dev(Q), dev(K)
    dense = torch.empty((b0, b1, s, s), device="cuda:0")
    tri = torch.empty((b0, b1, s, s), device="cuda:0")

    def calls():
        for out, causal in ((dense, 0), (tri, rp.CAUSAL_OUTPUT)):
            rp.bmm_raw(b0, b1, s, s, k, dQ, b1 * s * k, s * k, k, 0, dK, b1 * s * k, s * k, k, 1,
                       alpha, out, b1 * s * s, s * s, s, launch=ring_launch(rp), causal=causal)

    lower = torch.tril(torch.ones((s, s), dtype=torch.bool, device="cuda:0"))
    announce("ring graph", "eager")
    calls()
    torch.cuda.synchronize()
    eager_dense = host(dense).copy()
    eager_tri = host(torch.where(lower, tri, torch.zeros_like(tri))).copy()
    assert_bits_equal(eager_dense, want, "ring eager dense scores")
    assert_bits_equal(eager_tri, np.where(np.tril(np.ones((s, s), bool)), want, np.float32(0)),
                      "ring eager lower-triangle scores")
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
        announce("ring graph", "replay", rep)
        dense.fill_(float("nan"))
        tri.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert_bits_equal(host(dense), eager_dense, f"ring graph dense replay {rep}")
        got_tri = host(torch.where(lower, tri, torch.zeros_like(tri)))
        assert_bits_equal(got_tri, eager_tri, f"ring graph lower-triangle replay {rep}")

"""A whole training step of the DistilBERT feed-forward block on the GPU --
forward, every gradient, the AdamW update of every parameter, two steps in a
row -- equals the same step composed from oracle calls, bit for bit.  This is
the property the dispute protocol relies on: a training step re-executed on
other hardware gives the same checkpoint."""
import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal
from gpu_util import announce, dev, host
from paper_2502_19405_amd import inputs

pytestmark = pytest.mark.gpu


def oracle_step(P, M, V, X, dY, step, lr=1e-4, b1=0.9, b2=0.999, eps=1e-8, wd=0.01):
    W1, bb1, W2, bb2, gam, bet = P
    H1 = oracle.matmul(X, W1, bb1)
    G = oracle.gelu(H1)
    H2 = oracle.matmul(G, W2, bb2)
    Y, mean, rstd = oracle.layernorm_rows(H2, gam, bet, eps=1e-5, with_stats=True)
    dH2, dgam, dbet = oracle.layernorm_backward_rows(H2, dY, mean, rstd, gam)
    dW2 = oracle.matmul(G, dH2, trans_a=True)
    db2 = oracle.colsum_rows(dH2)
    dG = oracle.matmul(dH2, W2, trans_b=True)
    dH1 = oracle.gelu_backward(H1, dG)
    dW1 = oracle.matmul(X, dH1, trans_a=True)
    db1 = oracle.colsum_rows(dH1)
    dX = oracle.matmul(dH1, W1, trans_b=True)
    grads = [dW1, db1, dW2, db2, dgam, dbet]
    flat = lambda ts: np.concatenate([t.ravel() for t in ts])  # noqa: E731
    p, m, v = oracle.adam_step(flat(P), flat(grads), M, V, lr, b1, b2, eps, wd, step, True)
    out, off = [], 0
    for t in P:
        out.append(p[off:off + t.size].reshape(t.shape))
        off += t.size
    return Y, dX, grads, out, m, v


@pytest.mark.parametrize("tokens", [256, 1024])
def test_mlp_training_step_is_bitwise_the_oracle(tokens):
    import torch
    from paper_2502_19405_amd import pipelines
    d = inputs.distilbert_mlp(tokens=tokens)
    g = inputs.rng(1100 + tokens)
    names = ("W1", "b1", "W2", "b2", "gamma", "beta")
    P = [d[k] for k in names]
    st = pipelines.MlpTrainState(*(dev(d[k]) for k in names))
    n = st.param.numel()
    M, V = np.zeros(n, np.float32), np.zeros(n, np.float32)
    Xd = dev(d["X"])
    for step in (1, 2):
        dY = inputs.normal(g, (tokens, 768), var=1e-4)
        announce("mlp train step", tokens, step)
        Yg, dXg = pipelines.mlp_train_step(st, Xd, dev(dY))
        torch.cuda.synchronize()
        Y, dX, grads, P, M, V = oracle_step(P, M, V, d["X"], dY, step)
        assert_bits_equal(host(Yg), Y, f"Y step {step}")
        assert_bits_equal(host(dXg), dX, f"dX step {step}")
        for name, gg, gw in zip(names, st.g, grads):
            assert_bits_equal(host(gg), gw, f"grad {name} step {step}")
        for name, pg, pw in zip(names, st.p, P):
            assert_bits_equal(host(pg), pw, f"param {name} step {step}")
        assert_bits_equal(host(st.exp_avg), M, f"exp_avg step {step}")
        assert_bits_equal(host(st.exp_avg_sq), V, f"exp_avg_sq step {step}")

"""Oracle compositions of the model-shaped programs.

TEST INFRASTRUCTURE ONLY, like the rest of this package: each function chains
oracle calls in the order the corresponding program runs them, with no
arithmetic of its own beyond slicing and concatenating arrays.  They state what
the GPU compositions must produce bit for bit:

  mlp_forward         DistilBERT feed-forward block (Section 4.2's DistilBERT
                      programs): LayerNorm(gelu(X W1 + b1) W2 + b2)
  attention_forward   causal multi-head self-attention of the Llama programs
                      (Section 4.2), heads read in place by the batched product
                      (Section 2.2's key-query products)
  linear_backward     the two backward products of a linear layer
  mlp_train_step      one training step of the feed-forward block: forward,
                      every gradient, AdamW over all parameters (Sections 2.1-2.2:
                      a training step is what the protocol re-executes)
"""
from __future__ import annotations

import math

import numpy as np

from . import (adam_step, bmm_raw, colsum_rows, gelu, gelu_backward, layernorm_backward_rows,
               layernorm_rows, matmul, softmax_rows)


def mlp_forward(X, W1, b1, W2, b2, gamma, beta, eps=1e-5, nthreads=0):
    H1 = matmul(X, W1, b1, nthreads=nthreads)
    G = gelu(H1, nthreads=nthreads)
    H2 = matmul(G, W2, b2, nthreads=nthreads)
    Y = layernorm_rows(H2, gamma, beta, eps=eps, nthreads=nthreads)
    return {"H1": H1, "G": G, "H2": H2, "Y": Y}


def attention_scale(head_dim: int) -> np.float32:
    """1/sqrt(head_dim) rounded once to binary32."""
    return np.float32(1.0 / math.sqrt(head_dim))


def attention_forward(X, Wq, Wk, Wv, Wo, batch, seq, heads, nthreads=0):
    """Q, K, V = X Wq, X Wk, X Wv; per (b, h): S = alpha Q_h K_h^T, P = causal
    softmax rows of S, O_h = P V_h written into O's head columns; out = O Wo."""
    d = X.shape[1]
    hd = d // heads
    alpha = attention_scale(hd)
    Q = matmul(X, Wq, nthreads=nthreads)
    K = matmul(X, Wk, nthreads=nthreads)
    V = matmul(X, Wv, nthreads=nthreads)
    S = np.empty((batch, heads, seq, seq), np.float32)
    bmm_raw(batch, heads, seq, seq, hd, Q, seq * d, hd, d, 0, K, seq * d, hd, d, 1, alpha,
            S, heads * seq * seq, seq * seq, seq, nthreads=nthreads)
    P = softmax_rows(S.reshape(batch * heads * seq, seq), causal_period=seq, nthreads=nthreads)
    O = np.empty((batch * seq, d), np.float32)
    bmm_raw(batch, heads, seq, hd, seq, P, heads * seq * seq, seq * seq, seq, 0,
            V, seq * d, hd, d, 0, 1.0, O, seq * d, hd, d, nthreads=nthreads)
    out = matmul(O, Wo, nthreads=nthreads)
    return {"Q": Q, "K": K, "V": V, "S": S, "P": P, "O": O, "out": out}


def linear_backward(X, dY, W, nthreads=0):
    """dX = dY W^T (contraction over the output features), dW = X^T dY
    (contraction over the tokens)."""
    dX = matmul(dY, W, trans_b=True, nthreads=nthreads)
    dW = matmul(X, dY, trans_a=True, nthreads=nthreads)
    return dX, dW


MLP_PARAM_NAMES = ("W1", "b1", "W2", "b2", "gamma", "beta")


def mlp_train_step(P, M, V, X, dY, step, lr=1e-4, b1=0.9, b2=0.999, eps=1e-8, wd=0.01,
                   ln_eps=1e-5, nthreads=0):
    """One step of the feed-forward block with loss gradient dY.  P: the six
    parameters (W1, b1, W2, b2, gamma, beta); M, V: flat Adam moments in the
    same order.  Returns (Y, dX, grads, new params, M, V)."""
    W1, bb1, W2, bb2, gam, bet = P
    H1 = matmul(X, W1, bb1, nthreads=nthreads)
    G = gelu(H1, nthreads=nthreads)
    H2 = matmul(G, W2, bb2, nthreads=nthreads)
    Y, mean, rstd = layernorm_rows(H2, gam, bet, eps=ln_eps, with_stats=True, nthreads=nthreads)
    dH2, dgam, dbet = layernorm_backward_rows(H2, dY, mean, rstd, gam, nthreads=nthreads)
    dW2 = matmul(G, dH2, trans_a=True, nthreads=nthreads)
    db2 = colsum_rows(dH2, nthreads=nthreads)
    dG = matmul(dH2, W2, trans_b=True, nthreads=nthreads)
    dH1 = gelu_backward(H1, dG, nthreads=nthreads)
    dW1 = matmul(X, dH1, trans_a=True, nthreads=nthreads)
    db1 = colsum_rows(dH1, nthreads=nthreads)
    dX = matmul(dH1, W1, trans_b=True, nthreads=nthreads)
    grads = [dW1, db1, dW2, db2, dgam, dbet]
    flat = lambda ts: np.concatenate([t.ravel() for t in ts])  # noqa: E731
    p, m, v = adam_step(flat(P), flat(grads), M, V, lr, b1, b2, eps, wd, step, True,
                        nthreads=nthreads)
    out, off = [], 0
    for t in P:
        out.append(p[off:off + t.size].reshape(t.shape))
        off += t.size
    return Y, dX, grads, out, m, v

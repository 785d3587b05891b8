"""Model-shaped compositions of the reproducible operators.

Each function only chains C-ABI calls through the binding (no arithmetic of
its own), in the shapes of the programs Verde's evaluation runs (Section 4.2):
a DistilBERT feed-forward block, a Llama attention block and the backward
products of a Llama linear layer.  The feed-forward GELU is produced by the
first product's epilogue (repops_matmul_gelu), and in the training step the
GELU's input gradient by the epilogue of the product that makes its output
gradient (repops_matmul_gelu_backward); both give the bits of the
product and of the elementwise operator taken separately.  Every other
intermediate comes from its own operator call.
"""
from __future__ import annotations

import math

import torch

from . import repops


def mlp_forward(X, W1, b1, W2, b2, gamma, beta, eps=1e-5, order=None, gemm_launch=None,
                keep=False):
    """LayerNorm(gelu(X W1 + b1) W2 + b2): X [t, h], W1 [h, f], W2 [f, h]."""
    H1, G = repops.matmul_gelu(X, W1, b1, order=order, launch=gemm_launch)
    H2 = repops.matmul(G, W2, b2, order=order, launch=gemm_launch)
    Y = repops.layernorm_rows(H2, gamma, beta, eps=eps, order=order)
    if keep:
        return {"H1": H1, "G": G, "H2": H2, "Y": Y}
    return Y


def attention_scale(head_dim: int) -> float:
    """The binary32 value nearest 1/sqrt(head_dim) (exact for powers of 4)."""
    return float(torch.tensor(1.0 / math.sqrt(head_dim), dtype=torch.float32).item())


def attention_forward(X, Wq, Wk, Wv, Wo, batch, seq, heads, order=None, gemm_launch=None,
                      keep=False, buffers=None, causal_products=True):
    """Causal multi-head self-attention, fp32:
        Q, K, V = X Wq, X Wk, X Wv            [batch*seq, d]
        S[b,h]  = alpha * Q_h K_h^T            (bmm reading Q, K in place)
        P       = causal row softmax of S
        O_h     = P[b,h] V_h                   (written in place into [batch*seq, d])
        out     = O Wo
    Heads are column blocks of width d/heads of the projections.  With
    causal_products the score product computes only the tiles the causal
    softmax reads (S above the diagonal is left unspecified) and the value
    product skips P's all-zero blocks; P and O keep their bits either way."""
    d = X.shape[1]
    hd = d // heads
    alpha = attention_scale(hd)
    bufs = buffers or {}
    if gemm_launch is None:  # the three projections in one launch
        Q, K, V = repops.matmul_grouped([(X, Wq, None, bufs.get("Q")), (X, Wk, None, bufs.get("K")),
                                         (X, Wv, None, bufs.get("V"))], order=order)
    else:
        Q = repops.matmul(X, Wq, order=order, launch=gemm_launch, out=bufs.get("Q"))
        K = repops.matmul(X, Wk, order=order, launch=gemm_launch, out=bufs.get("K"))
        V = repops.matmul(X, Wv, order=order, launch=gemm_launch, out=bufs.get("V"))
    S = bufs.get("S")
    if S is None:
        S = torch.empty((batch, heads, seq, seq), dtype=torch.float32, device=X.device)
    # S[b,h] = Q[b*seq:(b+1)*seq, h*hd:(h+1)*hd] . K[...]^T
    repops.bmm_raw(batch, heads, seq, seq, hd,
                   Q, seq * d, hd, d, 0,
                   K, seq * d, hd, d, 1, alpha,
                   S, heads * seq * seq, seq * seq, seq, order=order, launch=gemm_launch,
                   causal=repops.CAUSAL_OUTPUT if causal_products else 0)
    P = repops.softmax_rows(S.view(batch * heads * seq, seq), causal_period=seq, order=order,
                            out=bufs.get("P"))
    O = bufs.get("O")
    if O is None:
        O = torch.empty((batch * seq, d), dtype=torch.float32, device=X.device)
    repops.bmm_raw(batch, heads, seq, hd, seq,
                   P, heads * seq * seq, seq * seq, seq, 0,
                   V, seq * d, hd, d, 0, 1.0,
                   O, seq * d, hd, d, order=order, launch=gemm_launch,
                   causal=repops.CAUSAL_A if causal_products else 0)
    out = repops.matmul(O, Wo, order=order, launch=gemm_launch, out=bufs.get("out"))
    if keep:
        return {"Q": Q, "K": K, "V": V, "S": S, "P": P, "O": O, "out": out}
    return out


def linear_backward(X, dY, W, order=None, gemm_launch=None, out_dx=None, out_dw=None):
    """Gradients of Y = X W: dX = dY W^T (contraction over the output
    features) and dW = X^T dY (contraction over the tokens); one grouped launch
    unless a launch configuration is given."""
    if gemm_launch is None:
        dX, dW = repops.matmul_grouped([(dY, W.t(), None, out_dx), (X.t(), dY, None, out_dw)],
                                       order=order)
        return dX, dW
    dX = repops.matmul(dY, W.t(), order=order, launch=gemm_launch, out=out_dx)
    dW = repops.matmul(X.t(), dY, order=order, launch=gemm_launch, out=out_dw)
    return dX, dW


class MlpTrainState:
    """Parameters, gradients and Adam moments of the feed-forward block in flat
    device buffers (one Adam launch updates everything); W1 [h, f], b1 [f],
    W2 [f, h], b2 [h], gamma [h], beta [h] are views into `param`, and the
    gradients are written straight into the matching views of `grad`."""

    def __init__(self, W1, b1, W2, b2, gamma, beta):
        h, f = W1.shape
        sizes = [h * f, f, f * h, h, h, h]
        self.shapes = [(h, f), (f,), (f, h), (h,), (h,), (h,)]
        n = sum(sizes)
        dev = W1.device
        self.param = torch.empty(n, dtype=torch.float32, device=dev)
        self.grad = torch.empty_like(self.param)
        self.exp_avg = torch.zeros_like(self.param)
        self.exp_avg_sq = torch.zeros_like(self.param)
        self.p, self.g = [], []
        off = 0
        for t, size, shape in zip((W1, b1, W2, b2, gamma, beta), sizes, self.shapes):
            self.p.append(self.param[off:off + size].view(shape))
            self.g.append(self.grad[off:off + size].view(shape))
            self.p[-1].copy_(t)
            off += size
        self.step = 0


def mlp_train_step(state: MlpTrainState, X, dY, lr=1e-4, betas=(0.9, 0.999), eps=1e-8,
                   weight_decay=0.01, ln_eps=1e-5, order=None, gemm_launch=None, bufs=None):
    """One training step of the feed-forward block Y = LayerNorm(gelu(X W1 + b1) W2 + b2)
    given the loss gradient dY: forward, backward (every gradient), AdamW update
    of all parameters.  Returns (Y, dX).  Every operation is a library call, so
    the step is bitwise reproducible."""
    W1, b1, W2, b2, gamma, beta = state.p
    gW1, gb1, gW2, gb2, ggamma, gbeta = state.g
    t, h = X.shape
    f = W1.shape[1]
    dev = X.device
    b = bufs if bufs is not None else {}

    def buf(name, *shape):
        # reused across steps while the shape stays; replaced when it changes
        t_ = b.get(name)
        if t_ is None or tuple(t_.shape) != shape or t_.device != dev:
            t_ = b[name] = torch.empty(shape, dtype=torch.float32, device=dev)
        return t_

    # forward (the LayerNorm statistics are the backward's saved tensors)
    H1, G = repops.matmul_gelu(X, W1, b1, order=order, launch=gemm_launch, out=buf("H1", t, f),
                               gelu_out=buf("G", t, f))
    H2 = repops.matmul(G, W2, b2, order=order, launch=gemm_launch, out=buf("H2", t, h))
    mean, rstd = buf("mean", t), buf("rstd", t)
    Y = repops.layernorm_rows(H2, gamma, beta, eps=ln_eps, order=order, out=buf("Y", t, h),
                              mean_out=mean, rstd_out=rstd)
    # backward.  dH1 = gelu_backward(H1, dH2 W2^T) straight from the product's
    # epilogue, alone: its 768 tiles make three even rounds over the compute
    # units.  Then both weight gradients (few output tiles, long contractions
    # over the tokens) and the input gradient dX run as one grouped launch, the
    # longest contractions first, so that dX's tiles fill the compute units the
    # weight gradients leave free.  (Grouping dW2 with dH1 instead measured 3%
    # slower per step.)  Every product keeps its own bits.
    dH2, _, _ = repops.layernorm_backward_rows(H2, dY, mean, rstd, gamma, order=order,
                                               dx_out=buf("dH2", t, h), dgamma_out=ggamma,
                                               dbeta_out=gbeta)
    dH1 = repops.matmul_gelu_backward(dH2, W2.t(), H1, order=order, launch=gemm_launch,
                                      out=buf("dH1", t, f))
    repops.colsum_rows(dH2, order=order, out=gb2)
    if gemm_launch is None:
        _, _, dX = repops.matmul_grouped([(G.t(), dH2, None, gW2), (X.t(), dH1, None, gW1),
                                          (dH1, W1.t(), None, buf("dX", t, h))], order=order)
    else:
        repops.matmul(G.t(), dH2, order=order, launch=gemm_launch, out=gW2)
        repops.matmul(X.t(), dH1, order=order, launch=gemm_launch, out=gW1)
        dX = repops.matmul(dH1, W1.t(), order=order, launch=gemm_launch, out=buf("dX", t, h))
    repops.colsum_rows(dH1, order=order, out=gb1)
    # optimizer
    state.step += 1
    repops.adam_step(state.param, state.grad, state.exp_avg, state.exp_avg_sq, lr, betas[0],
                     betas[1], eps, weight_decay, state.step, decoupled=True, order=order)
    return Y, dX

"""Seeded synthetic inputs for the RepOps operators.

This module only draws random numbers; it holds none of the operators'
arithmetic, so both the GPU path and the CPU oracle can be fed from it.  All
arrays are host numpy float32, C-contiguous, drawn from numpy's PCG64 generator
in the order the tensors are listed.  ``N(mu, var)`` takes a variance:
N(0, 4) draws with standard deviation 2, N(0, 0.02^2) with 0.02.

Workloads (shapes and distributions of the DistilBERT and Llama programs the
paper evaluates in Section 4.2; no trained weights or datasets are involved):

  gemm256_softmax256      A, B [256x256] ~ N(0,1); S [256x256] ~ N(0,4)
  gemm2048_bias           A, B [2048x2048] ~ U(-1,1); bias [2048] ~ U(-0.1,0.1)
  gemm2048_int            A, B [2048x2048], bias [2048]: integers in [-8, 8]
  distilbert_mlp          X [4096x768] ~ N(0,1); W1 [768x3072], W2 [3072x768]
                          ~ N(0, 0.02^2); b1, b2, beta ~ U(-0.1,0.1);
                          gamma = 1 + U(-0.1,0.1)
  llama_attention         X [4096x4096] ~ N(0,1) (batch 4 x seq 1024);
                          Wq, Wk, Wv, Wo [4096x4096] ~ N(0, 0.02^2)
  llama_linear_backward   X [8192x4096] ~ N(0,1); dY [8192x14336] ~ N(0, 1e-2);
                          W [4096x14336] ~ N(0, 0.02^2)
"""
from __future__ import annotations

import numpy as np

SEEDS = {
    "gemm256_softmax256": 0,
    "gemm2048_bias": 1,
    "gemm2048_int": 2,
    "distilbert_mlp": 3,
    "llama_attention": 4,
    "llama_linear_backward": 5,
}


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def normal(g: np.random.Generator, shape, var: float = 1.0) -> np.ndarray:
    """N(0, var) as float32 (drawn in float64, rounded once)."""
    return (g.standard_normal(shape) * np.sqrt(var)).astype(np.float32)


def uniform(g: np.random.Generator, shape, lo: float, hi: float) -> np.ndarray:
    return g.uniform(lo, hi, shape).astype(np.float32)


def integers(g: np.random.Generator, shape, lo: int = -8, hi: int = 8) -> np.ndarray:
    """Uniform integers in [lo, hi], stored as float32 (exact)."""
    return g.integers(lo, hi + 1, shape).astype(np.float32)


def gemm256_softmax256(seed: int = SEEDS["gemm256_softmax256"]):
    g = rng(seed)
    A = normal(g, (256, 256))
    B = normal(g, (256, 256))
    S = normal(g, (256, 256), var=4.0)
    return {"A": A, "B": B, "S": S}


def gemm2048_bias(seed: int = SEEDS["gemm2048_bias"], n: int = 2048):
    g = rng(seed)
    A = uniform(g, (n, n), -1.0, 1.0)
    B = uniform(g, (n, n), -1.0, 1.0)
    bias = uniform(g, (n,), -0.1, 0.1)
    return {"A": A, "B": B, "bias": bias}


def gemm2048_int(seed: int = SEEDS["gemm2048_int"], n: int = 2048):
    g = rng(seed)
    A = integers(g, (n, n))
    B = integers(g, (n, n))
    bias = integers(g, (n,))
    return {"A": A, "B": B, "bias": bias}


def distilbert_mlp(seed: int = SEEDS["distilbert_mlp"], tokens: int = 4096, hidden: int = 768,
                   ffn: int = 3072):
    g = rng(seed)
    X = normal(g, (tokens, hidden))
    W1 = normal(g, (hidden, ffn), var=0.02 ** 2)
    W2 = normal(g, (ffn, hidden), var=0.02 ** 2)
    b1 = uniform(g, (ffn,), -0.1, 0.1)
    b2 = uniform(g, (hidden,), -0.1, 0.1)
    gamma = (1.0 + g.uniform(-0.1, 0.1, (hidden,))).astype(np.float32)
    beta = uniform(g, (hidden,), -0.1, 0.1)
    return {"X": X, "W1": W1, "W2": W2, "b1": b1, "b2": b2, "gamma": gamma, "beta": beta}


def llama_attention(seed: int = SEEDS["llama_attention"], batch: int = 4, seq: int = 1024,
                    d_model: int = 4096):
    g = rng(seed)
    X = normal(g, (batch * seq, d_model))
    W = {name: normal(g, (d_model, d_model), var=0.02 ** 2) for name in ("Wq", "Wk", "Wv", "Wo")}
    return {"X": X, **W}


def llama_linear_backward(seed: int = SEEDS["llama_linear_backward"], tokens: int = 8192,
                          d_in: int = 4096, d_out: int = 14336):
    g = rng(seed)
    X = normal(g, (tokens, d_in))
    dY = normal(g, (tokens, d_out), var=1e-2)
    W = normal(g, (d_in, d_out), var=0.02 ** 2)
    return {"X": X, "dY": dY, "W": W}


def sample_indices(seed: int, npts: int, *extents: int):
    """npts index tuples drawn uniformly over the given extents, plus the
    corners (first and last index of every extent)."""
    g = rng(1000 + seed)
    cols = [g.integers(0, e, npts) for e in extents]
    corners = np.array(np.meshgrid(*[[0, e - 1] for e in extents], indexing="ij")).reshape(
        len(extents), -1)
    return tuple(np.concatenate([c, k]).astype(np.int64) for c, k in zip(cols, corners))

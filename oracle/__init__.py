"""CPU oracle for the RepOps operators (Verde, arXiv 2502.19405, Section 3).

TEST INFRASTRUCTURE ONLY.  The oracle is a plain scalar-C statement of each
reproducible operator (``repops_ref.c``), loaded here through ctypes on numpy
arrays.  Only the test suite, the smoke check and the benchmark's CPU-baseline
leg import this package; the GPU library and its binding never do, and the two
share no code.  Every function takes and returns host numpy float32 arrays.

Parity status per function (details in the test docstrings):
  dot / matmul / bmm   pinned: integer closed forms, order witnesses, exact
                       rational brute force, error bound, layout invariance
  rowsum               pinned: order witness, integer rows, W=1 reduction
  exp / gelu           pinned: special values, accuracy bounds against
                       high-precision references, constants against definitions
  softmax / layernorm  pinned: closed-form rows, bounds against float64
  training, Llama-block, erf and commitment operators: pinned in their own
                       test modules (tests/test_oracle_*.py)

``oracle.compose`` chains these calls into the model-shaped programs (the
feed-forward block, its training step, causal attention, a linear layer's
backward products); ``tests/golden/make_oracle_digests.py`` records digests of
their full outputs at the large shapes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "repops_ref.c")
LIB_PATH = os.path.join(_HERE, "librepops_ref.so")

# Strict IEEE binary32 on the host: no contraction of a*b+c, no fast-math, SSE
# arithmetic without excess precision; -mfma lets fmaf() become one instruction.
CFLAGS = [
    "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-mfma",
    "-fexcess-precision=standard", "-fPIC", "-shared", "-Wall",
]

INNER_FMA, INNER_MUL_ADD = 0, 1
ROW_TREE, ROW_BLOCKED = 0, 1


def build(opt: str = "-O2", out: str | None = None) -> str:
    """Compile the oracle with gcc; returns the library path."""
    out = out or LIB_PATH
    flags = [f if f != "-O2" else opt for f in CFLAGS]
    tmp = out + ".tmp"
    cmd = ["gcc", *flags, "-o", tmp, _SRC, "-lm", "-lpthread"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


_lib = None
_f32p = ctypes.POINTER(ctypes.c_float)
_i64p = ctypes.POINTER(ctypes.c_int64)
_i64 = ctypes.c_int64
_int = ctypes.c_int
_flt = ctypes.c_float


def _declare(lib):
    sig = {
        "repops_ref_env_check": (_int, []),
        "repops_ref_default_threads": (_int, []),
        "repops_ref_dot": (_flt, [_i64, _int, _i64, _f32p, _i64, _f32p, _i64]),
        "repops_ref_matmul": (_int, [_i64, _int, _i64, _i64, _i64, _f32p, _i64, _int,
                                     _f32p, _i64, _int, _f32p, _f32p, _i64, _int]),
        "repops_ref_matmul_at": (_int, [_i64, _int, _i64, _i64, _i64, _f32p, _i64, _int,
                                        _f32p, _i64, _int, _f32p, _i64, _i64p, _i64p, _f32p]),
        "repops_ref_bmm": (_int, [_i64, _int, _i64, _i64, _i64, _i64, _i64,
                                  _f32p, _i64, _i64, _i64, _int,
                                  _f32p, _i64, _i64, _i64, _int,
                                  _flt, _f32p, _i64, _i64, _i64, _int]),
        "repops_ref_bmm_at": (_int, [_i64, _int, _i64, _i64, _i64, _i64, _i64,
                                     _f32p, _i64, _i64, _i64, _int,
                                     _f32p, _i64, _i64, _i64, _int,
                                     _flt, _i64, _i64p, _i64p, _i64p, _i64p, _f32p]),
        "repops_ref_rowsum": (_flt, [_int, _int, _i64, _f32p, _int]),
        "repops_ref_exp1": (_flt, [_flt]),
        "repops_ref_gelu1": (_flt, [_flt]),
        "repops_ref_exp": (_int, [_i64, _f32p, _f32p, _int]),
        "repops_ref_gelu": (_int, [_i64, _f32p, _f32p, _int]),
        "repops_ref_softmax_rows": (_int, [_int, _int, _i64, _i64, _f32p, _i64, _f32p, _i64,
                                           _i64, _int]),
        "repops_ref_layernorm_rows": (_int, [_int, _int, _i64, _i64, _f32p, _i64, _f32p, _f32p,
                                             _flt, _f32p, _i64, _f32p, _f32p, _int]),
    }
    sig.update({
        "repops_ref_softmax_backward_rows": (_int, [_int, _int, _i64, _i64, _f32p, _i64, _f32p,
                                                    _i64, _f32p, _i64, _i64, _int]),
        "repops_ref_layernorm_backward_rows": (_int, [_int, _int, _i64, _i64, _i64, _f32p, _i64,
                                                      _f32p, _i64, _f32p, _f32p, _f32p, _f32p,
                                                      _i64, _f32p, _f32p, _int]),
        "repops_ref_colsum_rows": (_int, [_i64, _i64, _i64, _f32p, _i64, _f32p, _int]),
        "repops_ref_gelu_grad1": (_flt, [_flt]),
        "repops_ref_gelu_backward": (_int, [_i64, _f32p, _f32p, _f32p, _int]),
        "repops_ref_adam_step": (_int, [_i64, _f32p, _f32p, _f32p, _f32p, _flt, _flt, _flt, _flt,
                                        _flt, _i64, _int, _int]),
        "repops_ref_adam_scalars": (_int, [_flt, _flt, _flt, _flt, _i64, _f32p]),
        "repops_ref_sincos1": (None, [_flt, _f32p, _f32p]),
        "repops_ref_sincos": (_int, [_i64, _f32p, _f32p, _f32p, _int]),
        "repops_ref_rope": (_int, [_i64, _i64, _i64, _f32p, _i64, _f32p, _i64, _i64, _int, _f32p,
                                   _i64, _int]),
        "repops_ref_rmsnorm_rows": (_int, [_int, _int, _i64, _i64, _f32p, _i64, _f32p, _flt,
                                           _f32p, _i64, _f32p, _int]),
        "repops_ref_rmsnorm_backward_rows": (_int, [_int, _int, _i64, _i64, _i64, _f32p, _i64,
                                                    _f32p, _i64, _f32p, _f32p, _f32p, _i64, _f32p,
                                                    _int]),
        "repops_ref_silu1": (_flt, [_flt]),
        "repops_ref_silu_grad1": (_flt, [_flt]),
        "repops_ref_silu": (_int, [_i64, _f32p, _f32p, _int]),
        "repops_ref_swiglu": (_int, [_i64, _f32p, _f32p, _f32p, _int]),
        "repops_ref_swiglu_backward": (_int, [_i64, _f32p, _f32p, _f32p, _f32p, _f32p, _int]),
        "repops_ref_erf1": (_flt, [_flt]),
        "repops_ref_gelu_erf1": (_flt, [_flt]),
        "repops_ref_gelu_erf_grad1": (_flt, [_flt]),
        "repops_ref_erf": (_int, [_i64, _f32p, _f32p, _int]),
        "repops_ref_gelu_erf": (_int, [_i64, _f32p, _f32p, _int]),
        "repops_ref_gelu_erf_backward": (_int, [_i64, _f32p, _f32p, _f32p, _int]),
        "repops_ref_sha256": (None, [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]),
        "repops_ref_commit": (_int, [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                     ctypes.c_void_p]),
    })
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


def load(path: str | None = None):
    """Load the oracle library, building it first if it is missing."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC):
            build()
        _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


def _p(a):
    if a is None:
        return None
    assert a.dtype == np.float32 and a.flags["C_CONTIGUOUS"], "oracle takes contiguous float32"
    return a.ctypes.data_as(_f32p)


def _pi(a):
    assert a.dtype == np.int64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(_i64p)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (code {rc})")


def env_check(lib=None) -> int:
    return (lib or load()).repops_ref_env_check()


def default_threads() -> int:
    return load().repops_ref_default_threads()


def dot(a, b, k_block=64, k_inner=INNER_FMA, lib=None) -> np.float32:
    a = np.ascontiguousarray(a, np.float32)
    b = np.ascontiguousarray(b, np.float32)
    assert a.shape == b.shape and a.ndim == 1
    return np.float32((lib or load()).repops_ref_dot(k_block, k_inner, a.size, _p(a), 1, _p(b), 1))


def _logical_dims(A, B, trans_a, trans_b):
    m, k = (A.shape[1], A.shape[0]) if trans_a else A.shape
    k2, n = (B.shape[1], B.shape[0]) if trans_b else B.shape
    assert k == k2, "inner dimensions differ"
    return m, n, k


def matmul(A, B, bias=None, trans_a=False, trans_b=False, k_block=64, k_inner=INNER_FMA,
           nthreads=0, lib=None):
    """C = A.B (+ bias) with A given as [M,K] (or [K,M] if trans_a) and B as
    [K,N] (or [N,K] if trans_b), contiguous; returns float32 [M,N]."""
    m, n, k = _logical_dims(A, B, trans_a, trans_b)
    C = np.empty((m, n), np.float32)
    rc = (lib or load()).repops_ref_matmul(k_block, k_inner, m, n, k, _p(A), A.shape[1],
                                           int(trans_a), _p(B), B.shape[1], int(trans_b),
                                           _p(bias), _p(C), n, nthreads)
    _check(rc, "matmul")
    return C


def matmul_at(A, B, rows, cols, bias=None, trans_a=False, trans_b=False, k_block=64,
              k_inner=INNER_FMA, lib=None):
    """The outputs C[rows[p], cols[p]] of matmul, computed one by one."""
    m, n, k = _logical_dims(A, B, trans_a, trans_b)
    rows = np.ascontiguousarray(rows, np.int64)
    cols = np.ascontiguousarray(cols, np.int64)
    out = np.empty(rows.size, np.float32)
    rc = (lib or load()).repops_ref_matmul_at(k_block, k_inner, m, n, k, _p(A), A.shape[1],
                                              int(trans_a), _p(B), B.shape[1], int(trans_b),
                                              _p(bias), rows.size, _pi(rows), _pi(cols), _p(out))
    _check(rc, "matmul_at")
    return out


def bmm_raw(batch0, batch1, m, n, k, A, sa0, sa1, lda, trans_a, B, sb0, sb1, ldb, trans_b,
            alpha, C, sc0, sc1, ldc, k_block=64, k_inner=INNER_FMA, nthreads=0, lib=None):
    """Strided batched product on flat float32 buffers (element strides)."""
    rc = (lib or load()).repops_ref_bmm(k_block, k_inner, batch0, batch1, m, n, k,
                                        _p(A), sa0, sa1, lda, int(trans_a),
                                        _p(B), sb0, sb1, ldb, int(trans_b),
                                        float(alpha), _p(C), sc0, sc1, ldc, nthreads)
    _check(rc, "bmm")
    return C


def bmm_at_raw(batch0, batch1, m, n, k, A, sa0, sa1, lda, trans_a, B, sb0, sb1, ldb, trans_b,
               alpha, b0, b1, rows, cols, k_block=64, k_inner=INNER_FMA, lib=None):
    b0, b1, rows, cols = (np.ascontiguousarray(v, np.int64) for v in (b0, b1, rows, cols))
    out = np.empty(rows.size, np.float32)
    rc = (lib or load()).repops_ref_bmm_at(k_block, k_inner, batch0, batch1, m, n, k,
                                           _p(A), sa0, sa1, lda, int(trans_a),
                                           _p(B), sb0, sb1, ldb, int(trans_b), float(alpha),
                                           rows.size, _pi(b0), _pi(b1), _pi(rows), _pi(cols),
                                           _p(out))
    _check(rc, "bmm_at")
    return out


def bmm(A, B, alpha=1.0, trans_a=False, trans_b=False, k_block=64, k_inner=INNER_FMA,
        nthreads=0, lib=None):
    """Contiguous batched product: A [b0,b1,M,K] (or [..,K,M]), B [b0,b1,K,N]
    (or [..,N,K]); returns [b0,b1,M,N] scaled by alpha."""
    b0, b1 = A.shape[:2]
    assert B.shape[:2] == (b0, b1)
    m, n, k = _logical_dims(A[0, 0], B[0, 0], trans_a, trans_b)
    C = np.empty((b0, b1, m, n), np.float32)
    return bmm_raw(b0, b1, m, n, k, A, A.shape[1] * A[0, 0].size, A[0, 0].size, A.shape[3],
                   trans_a, B, B.shape[1] * B[0, 0].size, B[0, 0].size, B.shape[3], trans_b,
                   alpha, C, b1 * m * n, m * n, n, k_block, k_inner, nthreads, lib)


def rowsum(x, row_width=64, row_combine=ROW_TREE, squares=False, lib=None) -> np.float32:
    x = np.ascontiguousarray(x, np.float32)
    return np.float32((lib or load()).repops_ref_rowsum(row_width, row_combine, x.size, _p(x),
                                                        int(squares)))


def exp1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_exp1(float(np.float32(x))))


def gelu1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_gelu1(float(np.float32(x))))


def exp(x, nthreads=0, lib=None):
    x = np.ascontiguousarray(x, np.float32)
    y = np.empty_like(x)
    _check((lib or load()).repops_ref_exp(x.size, _p(x), _p(y), nthreads), "exp")
    return y


def gelu(x, nthreads=0, lib=None):
    x = np.ascontiguousarray(x, np.float32)
    y = np.empty_like(x)
    _check((lib or load()).repops_ref_gelu(x.size, _p(x), _p(y), nthreads), "gelu")
    return y


def softmax_rows(X, causal_period=0, row_width=64, row_combine=ROW_TREE, nthreads=0, lib=None):
    X = np.ascontiguousarray(X, np.float32)
    rows, cols = X.shape
    Y = np.empty_like(X)
    rc = (lib or load()).repops_ref_softmax_rows(row_width, row_combine, rows, cols, _p(X), cols,
                                                 _p(Y), cols, causal_period, nthreads)
    _check(rc, "softmax_rows")
    return Y


def layernorm_rows(X, gamma=None, beta=None, eps=1e-5, row_width=64, row_combine=ROW_TREE,
                   nthreads=0, lib=None, with_stats=False):
    X = np.ascontiguousarray(X, np.float32)
    rows, cols = X.shape
    Y = np.empty_like(X)
    mean = np.empty(rows, np.float32)
    rstd = np.empty(rows, np.float32)
    rc = (lib or load()).repops_ref_layernorm_rows(row_width, row_combine, rows, cols, _p(X), cols,
                                                   _p(gamma), _p(beta), float(np.float32(eps)),
                                                   _p(Y), cols, _p(mean), _p(rstd), nthreads)
    _check(rc, "layernorm_rows")
    return (Y, mean, rstd) if with_stats else Y


# --------------------------------------------------------------------------
# training-step operators
# --------------------------------------------------------------------------

def softmax_backward_rows(Y, dY, causal_period=0, row_width=64, row_combine=ROW_TREE,
                          nthreads=0, lib=None):
    Y = np.ascontiguousarray(Y, np.float32)
    dY = np.ascontiguousarray(dY, np.float32)
    rows, cols = Y.shape
    dX = np.empty_like(Y)
    rc = (lib or load()).repops_ref_softmax_backward_rows(row_width, row_combine, rows, cols,
                                                          _p(Y), cols, _p(dY), cols, _p(dX), cols,
                                                          causal_period, nthreads)
    _check(rc, "softmax_backward_rows")
    return dX


def layernorm_backward_rows(X, dY, mean, rstd, gamma=None, row_width=64, row_combine=ROW_TREE,
                            k_block=64, want_dx=True, want_params=True, nthreads=0, lib=None):
    """Returns (dX, dgamma, dbeta); entries not requested are None."""
    X = np.ascontiguousarray(X, np.float32)
    dY = np.ascontiguousarray(dY, np.float32)
    rows, cols = X.shape
    dX = np.empty_like(X) if want_dx else None
    dg = np.empty(cols, np.float32) if want_params else None
    db = np.empty(cols, np.float32) if want_params else None
    rc = (lib or load()).repops_ref_layernorm_backward_rows(
        row_width, row_combine, k_block, rows, cols, _p(X), cols, _p(dY), cols,
        _p(np.ascontiguousarray(mean, np.float32)), _p(np.ascontiguousarray(rstd, np.float32)),
        _p(gamma), _p(dX), cols, _p(dg), _p(db), nthreads)
    _check(rc, "layernorm_backward_rows")
    return dX, dg, db


def colsum_rows(X, k_block=64, nthreads=0, lib=None):
    """Column sums over rows with the contraction rule (a linear layer's bias gradient)."""
    X = np.ascontiguousarray(X, np.float32)
    rows, cols = X.shape
    out = np.empty(cols, np.float32)
    _check((lib or load()).repops_ref_colsum_rows(k_block, rows, cols, _p(X), cols, _p(out),
                                                  nthreads), "colsum_rows")
    return out


def gelu_grad1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_gelu_grad1(float(np.float32(x))))


def gelu_backward(x, dy, nthreads=0, lib=None):
    x = np.ascontiguousarray(x, np.float32)
    dy = np.ascontiguousarray(dy, np.float32)
    dx = np.empty_like(x)
    _check((lib or load()).repops_ref_gelu_backward(x.size, _p(x), _p(dy), _p(dx), nthreads),
           "gelu_backward")
    return dx


def adam_step(param, grad, exp_avg, exp_avg_sq, lr, beta1=0.9, beta2=0.999, eps=1e-8,
              weight_decay=0.0, step=1, decoupled=False, nthreads=0, lib=None):
    """In place on copies: returns (param, exp_avg, exp_avg_sq) after one step."""
    p = np.array(param, np.float32, copy=True)
    m = np.array(exp_avg, np.float32, copy=True)
    v = np.array(exp_avg_sq, np.float32, copy=True)
    g = np.ascontiguousarray(grad, np.float32)
    rc = (lib or load()).repops_ref_adam_step(p.size, _p(p), _p(g), _p(m), _p(v),
                                              *(float(np.float32(a)) for a in
                                                (lr, beta1, beta2, eps, weight_decay)),
                                              int(step), int(decoupled), nthreads)
    _check(rc, "adam_step")
    return p, m, v


def adam_scalars(lr, beta1, beta2, weight_decay, step, lib=None):
    out = np.empty(6, np.float32)
    rc = (lib or load()).repops_ref_adam_scalars(*(float(np.float32(a)) for a in
                                                   (lr, beta1, beta2, weight_decay)),
                                                 int(step), _p(out))
    _check(rc, "adam_scalars")
    return out


# --------------------------------------------------------------------------
# Llama-block operators
# --------------------------------------------------------------------------

def sincos1(x, lib=None):
    s, c = ctypes.c_float(), ctypes.c_float()
    (lib or load()).repops_ref_sincos1(float(np.float32(x)), ctypes.byref(s), ctypes.byref(c))
    return np.float32(s.value), np.float32(c.value)


def sincos(x, nthreads=0, lib=None):
    x = np.ascontiguousarray(x, np.float32)
    s, c = np.empty_like(x), np.empty_like(x)
    _check((lib or load()).repops_ref_sincos(x.size, _p(x), _p(s), _p(c), nthreads), "sincos")
    return s, c


def rope(X, heads, head_dim, inv_freq, period=0, offset=0, inverse=False, nthreads=0, lib=None):
    """X [rows, heads * head_dim] (contiguous); returns the rotated copy."""
    X = np.ascontiguousarray(X, np.float32)
    rows = X.shape[0]
    Y = np.empty_like(X)
    rc = (lib or load()).repops_ref_rope(rows, heads, head_dim, _p(X), X.shape[1],
                                         _p(np.ascontiguousarray(inv_freq, np.float32)), period,
                                         offset, int(inverse), _p(Y), X.shape[1], nthreads)
    _check(rc, "rope")
    return Y


def rmsnorm_rows(X, gamma=None, eps=1e-5, row_width=64, row_combine=ROW_TREE, nthreads=0,
                 lib=None, with_stats=False):
    X = np.ascontiguousarray(X, np.float32)
    rows, cols = X.shape
    Y = np.empty_like(X)
    rstd = np.empty(rows, np.float32)
    rc = (lib or load()).repops_ref_rmsnorm_rows(row_width, row_combine, rows, cols, _p(X), cols,
                                                 _p(gamma), float(np.float32(eps)), _p(Y), cols,
                                                 _p(rstd), nthreads)
    _check(rc, "rmsnorm_rows")
    return (Y, rstd) if with_stats else Y


def rmsnorm_backward_rows(X, dY, rstd, gamma=None, row_width=64, row_combine=ROW_TREE,
                          k_block=64, want_dx=True, want_params=True, nthreads=0, lib=None):
    """Returns (dX, dgamma); entries not requested are None."""
    X = np.ascontiguousarray(X, np.float32)
    dY = np.ascontiguousarray(dY, np.float32)
    rows, cols = X.shape
    dX = np.empty_like(X) if want_dx else None
    dg = np.empty(cols, np.float32) if want_params else None
    rc = (lib or load()).repops_ref_rmsnorm_backward_rows(
        row_width, row_combine, k_block, rows, cols, _p(X), cols, _p(dY), cols,
        _p(np.ascontiguousarray(rstd, np.float32)), _p(gamma), _p(dX), cols, _p(dg), nthreads)
    _check(rc, "rmsnorm_backward_rows")
    return dX, dg


def silu1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_silu1(float(np.float32(x))))


def silu_grad1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_silu_grad1(float(np.float32(x))))


def silu(x, nthreads=0, lib=None):
    x = np.ascontiguousarray(x, np.float32)
    y = np.empty_like(x)
    _check((lib or load()).repops_ref_silu(x.size, _p(x), _p(y), nthreads), "silu")
    return y


def swiglu(g, u, nthreads=0, lib=None):
    g = np.ascontiguousarray(g, np.float32)
    u = np.ascontiguousarray(u, np.float32)
    y = np.empty_like(g)
    _check((lib or load()).repops_ref_swiglu(g.size, _p(g), _p(u), _p(y), nthreads), "swiglu")
    return y


def swiglu_backward(g, u, dy, nthreads=0, lib=None):
    g = np.ascontiguousarray(g, np.float32)
    u = np.ascontiguousarray(u, np.float32)
    dy = np.ascontiguousarray(dy, np.float32)
    dg, du = np.empty_like(g), np.empty_like(g)
    _check((lib or load()).repops_ref_swiglu_backward(g.size, _p(g), _p(u), _p(dy), _p(dg),
                                                      _p(du), nthreads), "swiglu_backward")
    return dg, du


def erf1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_erf1(float(np.float32(x))))


def gelu_erf1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_gelu_erf1(float(np.float32(x))))


def gelu_erf_grad1(x, lib=None) -> np.float32:
    return np.float32((lib or load()).repops_ref_gelu_erf_grad1(float(np.float32(x))))


def _unary(fn, x, nthreads, lib):
    x = np.ascontiguousarray(x, np.float32)
    y = np.empty_like(x)
    _check(getattr(lib or load(), fn)(x.size, _p(x), _p(y), nthreads), fn)
    return y


def erf(x, nthreads=0, lib=None):
    return _unary("repops_ref_erf", x, nthreads, lib)


def gelu_erf(x, nthreads=0, lib=None):
    return _unary("repops_ref_gelu_erf", x, nthreads, lib)


def gelu_erf_backward(x, dy, nthreads=0, lib=None):
    x = np.ascontiguousarray(x, np.float32)
    dy = np.ascontiguousarray(dy, np.float32)
    dx = np.empty_like(x)
    _check((lib or load()).repops_ref_gelu_erf_backward(x.size, _p(x), _p(dy), _p(dx), nthreads),
           "gelu_erf_backward")
    return dx


# --------------------------------------------------------------------------
# tensor commitments
# --------------------------------------------------------------------------

def _bytes_of(data):
    if isinstance(data, (bytes, bytearray)):
        return np.frombuffer(bytes(data), np.uint8)
    return np.ascontiguousarray(data).view(np.uint8).ravel()


def sha256(data, lib=None) -> bytes:
    b = _bytes_of(data)
    out = (ctypes.c_uint8 * 32)()
    (lib or load()).repops_ref_sha256(b.ctypes.data if b.size else None, b.size, out)
    return bytes(out)


def commit(data, chunk_bytes=1024, lib=None) -> bytes:
    """RFC 6962 Merkle Tree Hash of the data's bytes in chunks of chunk_bytes."""
    b = _bytes_of(data)
    out = (ctypes.c_uint8 * 32)()
    _check((lib or load()).repops_ref_commit(b.ctypes.data if b.size else None, b.size,
                                             chunk_bytes, out), "commit")
    return bytes(out)

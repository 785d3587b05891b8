"""Python binding of librepops (ctypes over the C ABI in include/repops.h).

Argument marshalling only: every step of every operator runs in the HIP
kernels of librepops.so.  torch supplies device memory (``data_ptr``) and the
current HIP stream; nothing here computes on tensor values.  If the library is
missing, every call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librepops.so")

(OK, ERR_NULL, ERR_SHAPE, ERR_STRIDE, ERR_ALIAS, ERR_ORDER, ERR_LAUNCH, ERR_HIP, ERR_VALUE,
 ERR_WORKSPACE, ERR_SCRATCH) = range(11)
NOALLOC_SCRATCH_BYTES = 8 << 20  # REPOPS_NOALLOC_SCRATCH_BYTES
K_FMA, K_MUL_ADD = 0, 1
ROW_STRIDED_TREE, ROW_BLOCKED_LTR = 0, 1
LAUNCH_AUTO = 0
LAUNCH_GEMM_SIMPLE, LAUNCH_GEMM_TILED, LAUNCH_GEMM_MFMA = 1, 2, 3
LAUNCH_ROWS_GENERIC, LAUNCH_ROWS_WAVE = 1, 2
LAUNCH_ELEMENTWISE = 1


class OrderT(ctypes.Structure):
    _fields_ = [("version", ctypes.c_uint32), ("k_block", ctypes.c_uint32),
                ("k_inner", ctypes.c_uint32), ("k_combine", ctypes.c_uint32),
                ("row_width", ctypes.c_uint32), ("row_combine", ctypes.c_uint32),
                ("reserved", ctypes.c_uint32 * 2)]


class LaunchT(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_uint32), ("p", ctypes.c_uint32 * 7)]


@dataclass(frozen=True)
class Order:
    """Canonical-order descriptor (selects the bits)."""
    k_block: int = 64
    k_inner: int = K_FMA
    row_width: int = 64
    row_combine: int = ROW_STRIDED_TREE
    version: int = 1
    k_combine: int = 0

    def c(self) -> OrderT:
        o = OrderT()
        o.version, o.k_block, o.k_inner = self.version, self.k_block, self.k_inner
        o.k_combine, o.row_width, o.row_combine = self.k_combine, self.row_width, self.row_combine
        return o


@dataclass(frozen=True)
class Launch:
    """Launch descriptor (selects the speed only)."""
    kind: int = LAUNCH_AUTO
    p: tuple = field(default_factory=tuple)

    def c(self) -> LaunchT:
        l = LaunchT()
        l.kind = self.kind
        for i, v in enumerate(self.p):
            l.p[i] = v
        return l


class RepopsError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {status_str(code)} (code {code})")


class GemmDescT(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64), ("k", ctypes.c_int64),
                ("A", ctypes.c_void_p), ("lda", ctypes.c_int64), ("trans_a", ctypes.c_int32),
                ("B", ctypes.c_void_p), ("ldb", ctypes.c_int64), ("trans_b", ctypes.c_int32),
                ("bias", ctypes.c_void_p), ("C", ctypes.c_void_p), ("ldc", ctypes.c_int64),
                ("gelu_in", ctypes.c_void_p), ("ld_gelu_in", ctypes.c_int64)]


MAX_GROUP = 8  # REPOPS_MAX_GROUP
CAUSAL_OUTPUT, CAUSAL_A = 1, 2  # repops_bmm_causal masks

_lib = None
_i64, _i32, _u32, _f32, _vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float, ctypes.c_void_p
_op, _lp = ctypes.POINTER(OrderT), ctypes.POINTER(LaunchT)

_SIGNATURES = {
    "repops_order_default": (None, [_op]),
    "repops_status_str": (ctypes.c_char_p, [_i32]),
    "repops_abi_version": (_u32, []),
    "repops_gemm_config_count": (_i32, [_u32]),
    "repops_gemm_config_name": (ctypes.c_char_p, [_u32, _u32]),
    "repops_matmul": (_i32, [_op, _i64, _i64, _i64, _vp, _i64, _i32, _vp, _i64, _i32, _vp, _vp,
                             _i64, _lp, _vp]),
    "repops_matmul_gelu": (_i32, [_op, _i64, _i64, _i64, _vp, _i64, _i32, _vp, _i64, _i32, _vp,
                                  _vp, _i64, _vp, _i64, _lp, _vp]),
    "repops_matmul_gelu_backward": (_i32, [_op, _i64, _i64, _i64, _vp, _i64, _i32, _vp, _i64, _i32,
                                           _vp, _i64, _vp, _i64, _lp, _vp]),
    "repops_matmul_grouped": (_i32, [_op, _i32, ctypes.POINTER(GemmDescT), _lp, _vp]),
    "repops_bmm_causal": (_i32, [_op, _i64, _i64, _i64, _i64, _i64, _vp, _i64, _i64, _i64, _i32,
                                 _vp, _i64, _i64, _i64, _i32, _f32, _vp, _i64, _i64, _i64, _i32,
                                 _lp, _vp]),
    "repops_bmm": (_i32, [_op, _i64, _i64, _i64, _i64, _i64, _vp, _i64, _i64, _i64, _i32,
                          _vp, _i64, _i64, _i64, _i32, _f32, _vp, _i64, _i64, _i64, _lp, _vp]),
    "repops_softmax_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _i64, _i64, _lp, _vp]),
    "repops_layernorm_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _vp, _f32, _vp, _i64, _vp,
                                     _vp, _lp, _vp]),
    "repops_gelu": (_i32, [_op, _i64, _vp, _vp, _lp, _vp]),
    "repops_exp": (_i32, [_op, _i64, _vp, _vp, _lp, _vp]),
    "repops_copy": (_i32, [_op, _i64, _vp, _vp, _lp, _vp]),
    "repops_softmax_backward_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _i64,
                                            _i64, _lp, _vp]),
    "repops_layernorm_backward_workspace": (_i32, [_op, _i64, _i64, ctypes.POINTER(ctypes.c_uint64)]),
    "repops_layernorm_backward_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _vp,
                                              _vp, _i64, _vp, _vp, _vp, ctypes.c_uint64, _lp, _vp]),
    "repops_layernorm_backward_rows_noalloc": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _i64, _vp,
                                                      _vp, _vp, _vp, _i64, _vp, _vp, _lp, _vp]),
    "repops_gelu_backward": (_i32, [_op, _i64, _vp, _vp, _vp, _lp, _vp]),
    "repops_colsum_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _vp, ctypes.c_uint64, _lp, _vp]),
    "repops_adam_step": (_i32, [_op, _i64, _vp, _vp, _vp, _vp, _f32, _f32, _f32, _f32, _f32, _i64,
                                _i32, _lp, _vp]),
    "repops_sincos": (_i32, [_op, _i64, _vp, _vp, _vp, _lp, _vp]),
    "repops_rope": (_i32, [_op, _i64, _i64, _i64, _vp, _i64, _vp, _i64, _i64, _i32, _vp, _i64,
                           _lp, _vp]),
    "repops_rmsnorm_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _f32, _vp, _i64, _vp, _lp,
                                   _vp]),
    "repops_rmsnorm_backward_workspace": (_i32, [_op, _i64, _i64, ctypes.POINTER(ctypes.c_uint64)]),
    "repops_rmsnorm_backward_rows": (_i32, [_op, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _vp,
                                            _i64, _vp, _vp, ctypes.c_uint64, _lp, _vp]),
    "repops_silu": (_i32, [_op, _i64, _vp, _vp, _lp, _vp]),
    "repops_swiglu": (_i32, [_op, _i64, _vp, _vp, _vp, _lp, _vp]),
    "repops_swiglu_backward": (_i32, [_op, _i64, _vp, _vp, _vp, _vp, _vp, _lp, _vp]),
    "repops_erf": (_i32, [_op, _i64, _vp, _vp, _lp, _vp]),
    "repops_gelu_erf": (_i32, [_op, _i64, _vp, _vp, _lp, _vp]),
    "repops_gelu_erf_backward": (_i32, [_op, _i64, _vp, _vp, _vp, _lp, _vp]),
    "repops_commit_workspace": (_i32, [ctypes.c_uint64, _u32, ctypes.POINTER(ctypes.c_uint64)]),
    "repops_commit": (_i32, [_vp, ctypes.c_uint64, _u32, _vp, _vp, ctypes.c_uint64, _lp, _vp]),
}
EXPORTS = tuple(_SIGNATURES)


def load(path: str | None = None):
    """Load librepops.so (built in-tree by ``paper_2502_19405_amd.build``)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"librepops.so not found at {p}: build it with "
                           "`python -m paper_2502_19405_amd.build` (no fallback exists)")
    lib = ctypes.CDLL(p)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def status_str(code: int) -> str:
    return load().repops_status_str(code).decode()


def abi_version() -> int:
    return load().repops_abi_version()


def gemm_configs(kind: int = LAUNCH_GEMM_TILED) -> list[str]:
    lib = load()
    return [lib.repops_gemm_config_name(kind, i).decode()
            for i in range(lib.repops_gemm_config_count(kind))]


_DEFAULT_ORDER = Order()


def _check(rc: int, what: str):
    if rc != OK:
        raise RepopsError(rc, what)


_F32 = torch.float32


def _dev(t: torch.Tensor, name: str):
    if t.dtype is not _F32:
        raise TypeError(f"{name} must be float32")
    if not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    return t.data_ptr()


def _vec(t, name: str, size: int):
    """Pointer of an optional contiguous [size] float32 device vector."""
    if t is None:
        return None
    if t.numel() != size or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous [{size}] tensor")
    return _dev(t, name)


def _workspace(t):
    """(pointer, bytes) of a caller's workspace: any contiguous device tensor,
    whose size the library checks against what the call needs."""
    if t is None:
        return None, 0
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor")
    return t.data_ptr(), t.numel() * t.element_size()


try:  # the raw handle of the current stream, without building a Stream object
    _raw_stream = torch._C._cuda_getCurrentRawStream
except AttributeError:  # pragma: no cover - older torch
    _raw_stream = None


def _stream(t: torch.Tensor):
    if _raw_stream is not None:
        return _raw_stream(t.get_device())
    return torch.cuda.current_stream(t.device).cuda_stream


def _mat(t: torch.Tensor, name: str):
    """(pointer, rows, cols, ld, transposed) of a 2-D tensor with unit stride in
    one dimension: a row-major view, or the transpose of one."""
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    r, c = t.shape
    s0, s1 = t.stride()
    if t.numel() == 0:
        return t.data_ptr(), r, c, max(c, 1), 0
    if s1 == 1 and (s0 >= max(c, 1) or r <= 1):
        return _dev(t, name), r, c, max(s0, c, 1), 0
    if s0 == 1 and (s1 >= max(r, 1) or c <= 1):
        return _dev(t, name), r, c, max(s1, r, 1), 1
    raise ValueError(f"{name}: needs unit stride along one dimension (got strides {t.stride()})")


_STRUCTS: dict = {}
_DEFAULT_REF: list = []  # the default descriptor's reference, once built


def _ord(order):
    """ctypes reference to the descriptor struct of `order` (default if None),
    built once per distinct descriptor."""
    if order is None and _DEFAULT_REF:
        return _DEFAULT_REF[0]
    o = order or _DEFAULT_ORDER
    r = _STRUCTS.get(o)
    if r is None:
        c = o.c()
        r = _STRUCTS[o] = (c, ctypes.byref(c))
    if order is None:
        _DEFAULT_REF.append(r[1])
    return r[1]


def _launch(launch):
    if launch is None:
        return None
    r = _STRUCTS.get(launch)
    if r is None:
        c = launch.c()
        r = _STRUCTS[launch] = (c, ctypes.byref(c))
    return r[1]


def matmul(A: torch.Tensor, B: torch.Tensor, bias: torch.Tensor | None = None,
           order: Order | None = None, launch: Launch | None = None,
           out: torch.Tensor | None = None) -> torch.Tensor:
    """C = A @ B (+ bias).  A [m,k] and B [k,n] may be row-major or transposed
    views (``x.t()`` of a row-major tensor); out must be row-major."""
    pa, m, k, lda, ta = _mat(A, "A")
    pb, k2, n, ldb, tb = _mat(B, "B")
    if k != k2:
        raise ValueError(f"inner dimensions differ: {k} vs {k2}")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    ldc = _rows_as(out, m, n, "out")
    pbias = None
    if bias is not None:
        if bias.shape != (n,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous [n] tensor")
        pbias = _dev(bias, "bias")
    rc = load().repops_matmul(_ord(order), m, n, k, pa, lda, ta,
                              pb, ldb, tb, pbias, _dev(out, "out"), ldc,
                              _launch(launch), _stream(out))
    _check(rc, "repops_matmul")
    return out


def matmul_gelu(A: torch.Tensor, B: torch.Tensor, bias: torch.Tensor | None = None,
                order: Order | None = None, launch: Launch | None = None,
                out: torch.Tensor | None = None, gelu_out: torch.Tensor | None = None):
    """(H, G) with H = A @ B (+ bias) and G = gelu(H) from one pass: H has the
    bits matmul gives and G the bits gelu gives for that H."""
    pa, m, k, lda, ta = _mat(A, "A")
    pb, k2, n, ldb, tb = _mat(B, "B")
    if k != k2:
        raise ValueError(f"inner dimensions differ: {k} vs {k2}")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    if gelu_out is None:
        gelu_out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    ldh = _rows_as(out, m, n, "out")
    ldg = _rows_as(gelu_out, m, n, "gelu_out")
    pbias = None
    if bias is not None:
        if bias.shape != (n,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous [n] tensor")
        pbias = _dev(bias, "bias")
    rc = load().repops_matmul_gelu(_ord(order), m, n, k, pa, lda, ta, pb, ldb, tb, pbias,
                                   _dev(out, "out"), ldh, _dev(gelu_out, "gelu_out"), ldg,
                                   _launch(launch), _stream(out))
    _check(rc, "repops_matmul_gelu")
    return out, gelu_out


def _gelu_in(X, m, n):
    """(pointer, leading dimension) of a GELU backward's forward input."""
    ld = _rows_as(X, m, n, "gelu_in")
    return _dev(X, "gelu_in"), ld


def matmul_gelu_backward(A: torch.Tensor, B: torch.Tensor, X: torch.Tensor,
                         order: Order | None = None, launch: Launch | None = None,
                         out: torch.Tensor | None = None) -> torch.Tensor:
    """gelu_backward(X, A @ B) from one pass: the bits of matmul followed by
    gelu_backward."""
    pa, m, k, lda, ta = _mat(A, "A")
    pb, k2, n, ldb, tb = _mat(B, "B")
    if k != k2:
        raise ValueError(f"inner dimensions differ: {k} vs {k2}")
    px, ldx = _gelu_in(X, m, n)
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    ldc = _rows_as(out, m, n, "out")
    rc = load().repops_matmul_gelu_backward(_ord(order), m, n, k, pa, lda, ta, pb, ldb, tb, px,
                                            ldx, _dev(out, "out"), ldc,
                                            _launch(launch), _stream(out))
    _check(rc, "repops_matmul_gelu_backward")
    return out


def matmul_grouped(products, order: Order | None = None) -> list:
    """Several independent products in one call: products is a list of
    (A, B, bias, out) or (A, B, bias, out, gelu_in) with the meaning of matmul's
    arguments (bias and out may be None) and of matmul_gelu_backward's X;
    returns the outputs.  Every output has the bits matmul (or
    matmul_gelu_backward) gives."""
    if len(products) > MAX_GROUP:
        raise ValueError(f"at most {MAX_GROUP} products per call")
    descs = (GemmDescT * max(len(products), 1))()
    outs = []
    for d, prod in zip(descs, products):
        A, B, bias, out = prod[:4]
        X = prod[4] if len(prod) > 4 else None
        pa, m, k, lda, ta = _mat(A, "A")
        pb, k2, n, ldb, tb = _mat(B, "B")
        if k != k2:
            raise ValueError(f"inner dimensions differ: {k} vs {k2}")
        if out is None:
            out = torch.empty((m, n), dtype=torch.float32, device=A.device)
        ldc = _rows_as(out, m, n, "out")
        pbias = None
        if bias is not None:
            if bias.shape != (n,) or not bias.is_contiguous():
                raise ValueError("bias must be a contiguous [n] tensor")
            pbias = _dev(bias, "bias")
        d.m, d.n, d.k = m, n, k
        d.A, d.lda, d.trans_a, d.B, d.ldb, d.trans_b = pa, lda, ta, pb, ldb, tb
        d.bias, d.C, d.ldc = pbias, _dev(out, "out"), ldc
        if X is not None:
            d.gelu_in, d.ld_gelu_in = _gelu_in(X, m, n)
        outs.append(out)
    rc = load().repops_matmul_grouped(_ord(order), len(products), descs, None,
                                      _stream(outs[0]) if outs else None)
    _check(rc, "repops_matmul_grouped")
    return outs


def bmm_raw(batch0: int, batch1: int, m: int, n: int, k: int,
            A: torch.Tensor, sa0: int, sa1: int, lda: int, trans_a: int,
            B: torch.Tensor, sb0: int, sb1: int, ldb: int, trans_b: int, alpha: float,
            C: torch.Tensor, sc0: int, sc1: int, ldc: int,
            a_offset: int = 0, b_offset: int = 0, c_offset: int = 0,
            order: Order | None = None, launch: Launch | None = None, causal: int = 0):
    """The C-ABI bmm on raw element strides over the storage of A, B, C
    (offsets in elements from each tensor's data pointer).  causal: 0 for
    repops_bmm, else repops_bmm_causal's mask (CAUSAL_OUTPUT, CAUSAL_A)."""
    if causal:
        rc = load().repops_bmm_causal(_ord(order), batch0, batch1, m, n, k,
                                      _dev(A, "A") + 4 * a_offset, sa0, sa1, lda, trans_a,
                                      _dev(B, "B") + 4 * b_offset, sb0, sb1, ldb, trans_b, alpha,
                                      _dev(C, "C") + 4 * c_offset, sc0, sc1, ldc, causal,
                                      _launch(launch), _stream(C))
        _check(rc, "repops_bmm_causal")
        return C
    rc = load().repops_bmm(_ord(order), batch0, batch1, m, n, k,
                           _dev(A, "A") + 4 * a_offset, sa0, sa1, lda, trans_a,
                           _dev(B, "B") + 4 * b_offset, sb0, sb1, ldb, trans_b, alpha,
                           _dev(C, "C") + 4 * c_offset, sc0, sc1, ldc, _launch(launch), _stream(C))
    _check(rc, "repops_bmm")
    return C


def bmm(A: torch.Tensor, B: torch.Tensor, alpha: float = 1.0, order: Order | None = None,
        launch: Launch | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """C[b0,b1] = alpha * A[b0,b1] @ B[b0,b1] for 4-D tensors [b0, b1, r, c]
    whose last two dimensions are row-major or transposed views."""
    if A.dim() != 4 or B.dim() != 4:
        raise ValueError("bmm takes 4-D tensors [batch0, batch1, rows, cols]")
    b0, b1, m, k = A.shape
    n = B.shape[3]
    if tuple(B.shape[:2]) != (b0, b1):
        raise ValueError("batch dimensions differ")
    if B.shape[2] != k:
        raise ValueError(f"inner dimensions differ: {k} vs {B.shape[2]}")
    if out is None:
        out = torch.empty((b0, b1, m, n), dtype=torch.float32, device=A.device)
    if out.dim() != 4 or tuple(out.shape) != (b0, b1, m, n) or out.stride(3) != 1:
        raise ValueError(f"out must be a [{b0}, {b1}, {m}, {n}] tensor, row-major in its last two "
                         "dimensions")
    if b0 == 0 or b1 == 0:
        return out
    _, _, _, lda, ta = _mat(A[0, 0], "A")
    _, _, _, ldb, tb = _mat(B[0, 0], "B")
    rc = load().repops_bmm(_ord(order), b0, b1, m, n, k,
                           _dev(A, "A"), A.stride(0), A.stride(1), lda, ta,
                           _dev(B, "B"), B.stride(0), B.stride(1), ldb, tb, float(alpha),
                           _dev(out, "out"), out.stride(0), out.stride(1),
                           out.stride(2) if m > 1 else max(n, 1), _launch(launch), _stream(out))
    _check(rc, "repops_bmm")
    return out


def _rows(X: torch.Tensor, name: str):
    """(rows, cols, ld) of a 2-D tensor with unit column stride.  ld is the row
    stride as it stands, so rows that overlap (a row stride below cols, as in an
    expanded view) reach the library, which rejects them; a single row's stride
    is never used and passes as cols."""
    sh, st = X.shape, X.stride()
    if len(sh) != 2 or st[1] != 1:
        raise ValueError(f"{name} must be a 2-D tensor with unit column stride")
    return sh[0], sh[1], st[0] if sh[0] > 1 else max(sh[1], 1)


def _rows_as(t: torch.Tensor, rows: int, cols: int, name: str) -> int:
    """Row stride of a 2-D tensor with unit column stride that must be exactly
    [rows, cols] (the library writes or reads that many rows through it)."""
    r, c, ld = _rows(t, name)
    if r != rows or c != cols:
        raise ValueError(f"{name} must be [{rows}, {cols}] (got [{r}, {c}])")
    return ld


def softmax_rows(X: torch.Tensor, causal_period: int = 0, order: Order | None = None,
                 launch: Launch | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    rows, cols, ldx = _rows(X, "X")
    if out is None:
        out = torch.empty_like(X, memory_format=torch.contiguous_format)
    ldy = _rows_as(out, rows, cols, "out")
    rc = (_lib or load()).repops_softmax_rows(_ord(order), rows, cols, _dev(X, "X"), ldx,
                                              _dev(out, "out"), ldy, causal_period,
                                              _launch(launch), _stream(out))
    _check(rc, "repops_softmax_rows")
    return out


def layernorm_rows(X: torch.Tensor, gamma: torch.Tensor | None = None,
                   beta: torch.Tensor | None = None, eps: float = 1e-5,
                   order: Order | None = None, launch: Launch | None = None,
                   out: torch.Tensor | None = None, mean_out: torch.Tensor | None = None,
                   rstd_out: torch.Tensor | None = None) -> torch.Tensor:
    rows, cols, ldx = _rows(X, "X")
    if out is None:
        out = torch.empty_like(X, memory_format=torch.contiguous_format)
    ldy = _rows_as(out, rows, cols, "out")
    rc = (_lib or load()).repops_layernorm_rows(
        _ord(order), rows, cols, _dev(X, "X"), ldx, _vec(gamma, "gamma", cols),
        _vec(beta, "beta", cols), float(eps), _dev(out, "out"), ldy,
        _vec(mean_out, "mean_out", rows),
        _vec(rstd_out, "rstd_out", rows), _launch(launch), _stream(out))
    _check(rc, "repops_layernorm_rows")
    return out


def _elementwise(fn_name: str, X: torch.Tensor, order, launch, out):
    if not X.is_contiguous():
        raise ValueError("X must be contiguous")
    if out is None:
        out = torch.empty_like(X)
    if not out.is_contiguous() or out.numel() != X.numel():
        raise ValueError("out must be contiguous with X's element count")
    rc = getattr(load(), fn_name)(_ord(order), X.numel(),
                                  _dev(X, "X"), _dev(out, "out"), _launch(launch), _stream(out))
    _check(rc, fn_name)
    return out


def gelu(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None,
         out: torch.Tensor | None = None) -> torch.Tensor:
    return _elementwise("repops_gelu", X, order, launch, out)


def copy(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None,
         out: torch.Tensor | None = None) -> torch.Tensor:
    """Y = X through the elementwise kernel (the streaming ceiling it reaches)."""
    return _elementwise("repops_copy", X, order, launch, out)


def exp(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None,
        out: torch.Tensor | None = None) -> torch.Tensor:
    return _elementwise("repops_exp", X, order, launch, out)


# ---------------------------------------------------------------------------
# training-step operators
# ---------------------------------------------------------------------------

def softmax_backward_rows(Y: torch.Tensor, dY: torch.Tensor, causal_period: int = 0,
                          order: Order | None = None, launch: Launch | None = None,
                          out: torch.Tensor | None = None) -> torch.Tensor:
    """dX = Y * (dY - rowsum(Y * dY)) from the forward output Y."""
    rows, cols, ldy = _rows(Y, "Y")
    r2, c2, lddy = _rows(dY, "dY")
    if (r2, c2) != (rows, cols):
        raise ValueError("Y and dY shapes differ")
    if out is None:
        out = torch.empty_like(Y, memory_format=torch.contiguous_format)
    lddx = _rows_as(out, rows, cols, "out")
    rc = load().repops_softmax_backward_rows(
        _ord(order), rows, cols, _dev(Y, "Y"), ldy,
        _dev(dY, "dY"), lddy, _dev(out, "out"), lddx, causal_period, _launch(launch), _stream(out))
    _check(rc, "repops_softmax_backward_rows")
    return out


def layernorm_backward_workspace(rows: int, cols: int, order: Order | None = None) -> int:
    """Bytes of workspace the LayerNorm backward needs for its parameter gradients."""
    n = ctypes.c_uint64(0)
    rc = load().repops_layernorm_backward_workspace(_ord(order),
                                                    rows, cols, ctypes.byref(n))
    _check(rc, "repops_layernorm_backward_workspace")
    return n.value


def layernorm_backward_rows(X: torch.Tensor, dY: torch.Tensor, mean: torch.Tensor,
                            rstd: torch.Tensor, gamma: torch.Tensor | None = None,
                            need_dx: bool = True, need_params: bool = True,
                            order: Order | None = None, launch: Launch | None = None,
                            dx_out: torch.Tensor | None = None,
                            dgamma_out: torch.Tensor | None = None,
                            dbeta_out: torch.Tensor | None = None,
                            workspace: torch.Tensor | None = None):
    """(dX, dgamma, dbeta) of the row LayerNorm from the forward's mean / rstd;
    entries not requested are None.  Outputs and the workspace are allocated
    here unless passed (the library checks the workspace's size)."""
    rows, cols, ldx = _rows(X, "X")
    r2, c2, lddy = _rows(dY, "dY")
    if (r2, c2) != (rows, cols):
        raise ValueError("X and dY shapes differ")
    for t, name in ((mean, "mean"), (rstd, "rstd")):
        if t.numel() != rows or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous [{rows}] tensor")
    pg = None
    if gamma is not None:
        if gamma.numel() != cols or not gamma.is_contiguous():
            raise ValueError(f"gamma must be a contiguous [{cols}] tensor")
        pg = _dev(gamma, "gamma")
    dx = dgamma = dbeta = None
    lddx = cols
    if need_dx:
        dx = dx_out if dx_out is not None else torch.empty_like(X, memory_format=torch.contiguous_format)
        lddx = _rows_as(dx, rows, cols, "dx_out")
    wptr, wbytes = None, 0
    if need_params:
        dgamma = dgamma_out if dgamma_out is not None else torch.empty(cols, dtype=torch.float32,
                                                                       device=X.device)
        dbeta = dbeta_out if dbeta_out is not None else torch.empty(cols, dtype=torch.float32,
                                                                    device=X.device)
        for t, name in ((dgamma, "dgamma_out"), (dbeta, "dbeta_out")):
            if t.numel() != cols or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous [{cols}] tensor")
        if workspace is None:
            need = layernorm_backward_workspace(rows, cols, order)
            if need:
                workspace = torch.empty(need // 4, dtype=torch.float32, device=X.device)
        wptr, wbytes = _workspace(workspace)
    ptr = lambda t, n: None if t is None else _dev(t, n)  # noqa: E731
    rc = load().repops_layernorm_backward_rows(
        _ord(order), rows, cols, _dev(X, "X"), ldx, _dev(dY, "dY"), lddy,
        _dev(mean, "mean"), _dev(rstd, "rstd"), pg, ptr(dx, "dX"), lddx, ptr(dgamma, "dgamma"),
        ptr(dbeta, "dbeta"), wptr, wbytes, _launch(launch), _stream(X))
    _check(rc, "repops_layernorm_backward_rows")
    return dx, dgamma, dbeta


def layernorm_backward_rows_noalloc(X: torch.Tensor, dY: torch.Tensor, mean: torch.Tensor,
                                    rstd: torch.Tensor, gamma: torch.Tensor | None,
                                    dx_out: torch.Tensor | None, dgamma_out: torch.Tensor | None,
                                    dbeta_out: torch.Tensor | None, order: Order | None = None,
                                    launch: Launch | None = None):
    """repops_layernorm_backward_rows_noalloc: the LayerNorm backward into the
    caller's outputs (any of them None to skip it), with the parameter
    gradients' partials in the library's fixed scratch array -- nothing is
    allocated here or in the library.  Calls that overlap on one device
    race on the scratch array."""
    rows, cols, ldx = _rows(X, "X")
    r2, c2, lddy = _rows(dY, "dY")
    if (r2, c2) != (rows, cols):
        raise ValueError("X and dY shapes differ")
    for t, name in ((mean, "mean"), (rstd, "rstd")):
        if t.numel() != rows or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous [{rows}] tensor")
    for t, name in ((gamma, "gamma"), (dgamma_out, "dgamma_out"), (dbeta_out, "dbeta_out")):
        if t is not None and (t.numel() != cols or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous [{cols}] tensor")
    lddx = cols
    if dx_out is not None:
        lddx = _rows_as(dx_out, rows, cols, "dx_out")
    ptr = lambda t, n: None if t is None else _dev(t, n)  # noqa: E731
    rc = load().repops_layernorm_backward_rows_noalloc(
        _ord(order), rows, cols, _dev(X, "X"), ldx, _dev(dY, "dY"), lddy,
        _dev(mean, "mean"), _dev(rstd, "rstd"), ptr(gamma, "gamma"), ptr(dx_out, "dX"), lddx,
        ptr(dgamma_out, "dgamma"), ptr(dbeta_out, "dbeta"), _launch(launch), _stream(X))
    _check(rc, "repops_layernorm_backward_rows_noalloc")
    return dx_out, dgamma_out, dbeta_out


def colsum_rows(X: torch.Tensor, order: Order | None = None, out: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None) -> torch.Tensor:
    """Column sums of X [rows, cols] over rows (a linear layer's bias gradient)."""
    rows, cols, ldx = _rows(X, "X")
    if out is None:
        out = torch.empty(cols, dtype=torch.float32, device=X.device)
    wptr, wbytes = None, 0
    if workspace is None:
        need = layernorm_backward_workspace(rows, cols, order)
        if need:
            workspace = torch.empty(need // 4, dtype=torch.float32, device=X.device)
    wptr, wbytes = _workspace(workspace)
    rc = load().repops_colsum_rows(_ord(order), rows, cols, _dev(X, "X") if rows else None, ldx,
                                   _flat(out, cols, "out"), wptr, wbytes, None, _stream(out))
    _check(rc, "repops_colsum_rows")
    return out


def gelu_backward(X: torch.Tensor, dY: torch.Tensor, order: Order | None = None,
                  launch: Launch | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """dX = dY * gelu'(X), elementwise over contiguous tensors."""
    if not X.is_contiguous() or not dY.is_contiguous() or dY.numel() != X.numel():
        raise ValueError("X and dY must be contiguous with equal element counts")
    if out is None:
        out = torch.empty_like(X)
    if not out.is_contiguous() or out.numel() != X.numel():
        raise ValueError("out must be contiguous with X's element count")
    rc = load().repops_gelu_backward(_ord(order), X.numel(),
                                     _dev(X, "X"), _dev(dY, "dY"), _dev(out, "out"),
                                     _launch(launch), _stream(out))
    _check(rc, "repops_gelu_backward")
    return out


def erf(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None,
        out: torch.Tensor | None = None) -> torch.Tensor:
    return _elementwise("repops_erf", X, order, launch, out)


def gelu_erf(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None,
             out: torch.Tensor | None = None) -> torch.Tensor:
    """x * Phi(x), the erf form of GELU."""
    return _elementwise("repops_gelu_erf", X, order, launch, out)


def gelu_erf_backward(X: torch.Tensor, dY: torch.Tensor, order: Order | None = None,
                      launch: Launch | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    if not X.is_contiguous() or not dY.is_contiguous() or dY.numel() != X.numel():
        raise ValueError("X and dY must be contiguous with equal element counts")
    if out is None:
        out = torch.empty_like(X)
    rc = load().repops_gelu_erf_backward(_ord(order), X.numel(), _dev(X, "X"), _dev(dY, "dY"),
                                         _flat(out, X.numel(), "out"), _launch(launch),
                                         _stream(out))
    _check(rc, "repops_gelu_erf_backward")
    return out


def adam_step(param: torch.Tensor, grad: torch.Tensor, exp_avg: torch.Tensor,
              exp_avg_sq: torch.Tensor, lr: float, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8, weight_decay: float = 0.0, step: int = 1,
              decoupled: bool = True, order: Order | None = None,
              launch: Launch | None = None) -> None:
    """One Adam / AdamW update of param, exp_avg and exp_avg_sq in place."""
    n = param.numel()
    for t, name in ((param, "param"), (grad, "grad"), (exp_avg, "exp_avg"),
                    (exp_avg_sq, "exp_avg_sq")):
        if not t.is_contiguous() or t.numel() != n:
            raise ValueError(f"{name} must be contiguous with {n} elements")
    rc = load().repops_adam_step(_ord(order), n,
                                 _dev(param, "param"), _dev(grad, "grad"),
                                 _dev(exp_avg, "exp_avg"), _dev(exp_avg_sq, "exp_avg_sq"),
                                 float(lr), float(beta1), float(beta2), float(eps),
                                 float(weight_decay), int(step), 1 if decoupled else 0,
                                 _launch(launch), _stream(param))
    _check(rc, "repops_adam_step")


# ---------------------------------------------------------------------------
# Llama-block operators
# ---------------------------------------------------------------------------

def _flat(t: torch.Tensor, n: int, name: str):
    if not t.is_contiguous() or t.numel() != n:
        raise ValueError(f"{name} must be contiguous with {n} elements")
    return _dev(t, name)


def sincos(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None):
    """(sin X, cos X) elementwise (the reproducible sin/cos inside the rotary
    embedding, exported for testing)."""
    n = X.numel()
    S, C = torch.empty_like(X), torch.empty_like(X)
    rc = load().repops_sincos(_ord(order), n, _flat(X, n, "X"), _dev(S, "S"), _dev(C, "C"),
                              _launch(launch), _stream(X))
    _check(rc, "repops_sincos")
    return S, C


def rope(X: torch.Tensor, heads: int, head_dim: int, inv_freq: torch.Tensor,
         position_period: int = 0, position_offset: int = 0, inverse: bool = False,
         order: Order | None = None, launch: Launch | None = None,
         out: torch.Tensor | None = None) -> torch.Tensor:
    """Rotary embedding of X [rows, >= heads * head_dim] (rotate-half pairs);
    row r sits at position (r % period if period else r) + offset."""
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be a 2-D tensor with unit column stride")
    rows = X.shape[0]
    if X.shape[1] < heads * head_dim:
        raise ValueError("X is narrower than heads * head_dim")
    if out is None:
        out = torch.empty((rows, heads * head_dim), dtype=torch.float32, device=X.device)
    if (out.dim() != 2 or out.stride(1) != 1 or out.shape[0] != rows
            or out.shape[1] < heads * head_dim):
        raise ValueError(f"out must be a 2-D tensor with unit column stride, {rows} rows and at "
                         f"least {heads * head_dim} columns")
    pinv = _flat(inv_freq, head_dim // 2, "inv_freq")
    rc = load().repops_rope(_ord(order), rows, heads, head_dim, _dev(X, "X"),
                            X.stride(0) if rows > 1 else X.shape[1], pinv, position_period,
                            position_offset, 1 if inverse else 0, _dev(out, "out"),
                            out.stride(0) if rows > 1 else out.shape[1],
                            _launch(launch), _stream(X))
    _check(rc, "repops_rope")
    return out


def rmsnorm_rows(X: torch.Tensor, gamma: torch.Tensor | None = None, eps: float = 1e-5,
                 order: Order | None = None, launch: Launch | None = None,
                 out: torch.Tensor | None = None,
                 rstd_out: torch.Tensor | None = None) -> torch.Tensor:
    rows, cols, ldx = _rows(X, "X")
    if out is None:
        out = torch.empty_like(X, memory_format=torch.contiguous_format)
    ldy = _rows_as(out, rows, cols, "out")
    pg = None if gamma is None else _flat(gamma, cols, "gamma")
    pr = None if rstd_out is None else _flat(rstd_out, rows, "rstd_out")
    rc = load().repops_rmsnorm_rows(_ord(order), rows, cols, _dev(X, "X"), ldx, pg, float(eps),
                                    _dev(out, "out"), ldy, pr, _launch(launch), _stream(out))
    _check(rc, "repops_rmsnorm_rows")
    return out


def rmsnorm_backward_workspace(rows: int, cols: int, order: Order | None = None) -> int:
    n = ctypes.c_uint64(0)
    rc = load().repops_rmsnorm_backward_workspace(_ord(order), rows, cols, ctypes.byref(n))
    _check(rc, "repops_rmsnorm_backward_workspace")
    return n.value


def rmsnorm_backward_rows(X: torch.Tensor, dY: torch.Tensor, rstd: torch.Tensor,
                          gamma: torch.Tensor | None = None, need_dx: bool = True,
                          need_dgamma: bool = True, order: Order | None = None,
                          launch: Launch | None = None, dx_out: torch.Tensor | None = None,
                          dgamma_out: torch.Tensor | None = None,
                          workspace: torch.Tensor | None = None):
    """(dX, dgamma) of the RMSNorm from the forward's rstd; entries not
    requested are None."""
    rows, cols, ldx = _rows(X, "X")
    r2, c2, lddy = _rows(dY, "dY")
    if (r2, c2) != (rows, cols):
        raise ValueError("X and dY shapes differ")
    prs = _flat(rstd, rows, "rstd")
    pg = None if gamma is None else _flat(gamma, cols, "gamma")
    dx = dgamma = None
    lddx = cols
    if need_dx:
        dx = dx_out if dx_out is not None else torch.empty_like(X, memory_format=torch.contiguous_format)
        lddx = _rows_as(dx, rows, cols, "dx_out")
    wptr, wbytes = None, 0
    if need_dgamma:
        dgamma = dgamma_out if dgamma_out is not None else torch.empty(cols, dtype=torch.float32,
                                                                       device=X.device)
        if workspace is None:
            need = rmsnorm_backward_workspace(rows, cols, order)
            if need:
                workspace = torch.empty(need // 4, dtype=torch.float32, device=X.device)
        wptr, wbytes = _workspace(workspace)
    rc = load().repops_rmsnorm_backward_rows(
        _ord(order), rows, cols, _dev(X, "X"), ldx, _dev(dY, "dY"), lddy, prs, pg,
        None if dx is None else _dev(dx, "dX"), lddx,
        None if dgamma is None else _flat(dgamma, cols, "dgamma"), wptr, wbytes,
        _launch(launch), _stream(X))
    _check(rc, "repops_rmsnorm_backward_rows")
    return dx, dgamma


def silu(X: torch.Tensor, order: Order | None = None, launch: Launch | None = None,
         out: torch.Tensor | None = None) -> torch.Tensor:
    return _elementwise("repops_silu", X, order, launch, out)


def swiglu(G: torch.Tensor, Up: torch.Tensor, order: Order | None = None,
           launch: Launch | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """silu(G) * Up elementwise."""
    n = G.numel()
    if out is None:
        out = torch.empty_like(G)
    rc = load().repops_swiglu(_ord(order), n, _flat(G, n, "G"), _flat(Up, n, "Up"),
                              _flat(out, n, "out"), _launch(launch), _stream(out))
    _check(rc, "repops_swiglu")
    return out


def swiglu_backward(G: torch.Tensor, Up: torch.Tensor, dY: torch.Tensor,
                    order: Order | None = None, launch: Launch | None = None,
                    dg_out: torch.Tensor | None = None, du_out: torch.Tensor | None = None):
    """(dG, dUp) of silu(G) * Up."""
    n = G.numel()
    dG = dg_out if dg_out is not None else torch.empty_like(G)
    dU = du_out if du_out is not None else torch.empty_like(G)
    rc = load().repops_swiglu_backward(_ord(order), n, _flat(G, n, "G"), _flat(Up, n, "Up"),
                                       _flat(dY, n, "dY"), _flat(dG, n, "dG"), _flat(dU, n, "dUp"),
                                       _launch(launch), _stream(G))
    _check(rc, "repops_swiglu_backward")
    return dG, dU


# ---------------------------------------------------------------------------
# tensor commitments
# ---------------------------------------------------------------------------

def commit_workspace(nbytes: int, chunk_bytes: int = 1024) -> int:
    n = ctypes.c_uint64(0)
    _check(load().repops_commit_workspace(nbytes, chunk_bytes, ctypes.byref(n)),
           "repops_commit_workspace")
    return n.value


def commit(t: torch.Tensor, chunk_bytes: int = 1024, digest: torch.Tensor | None = None,
           workspace: torch.Tensor | None = None) -> torch.Tensor:
    """RFC 6962 Merkle commitment of a contiguous device tensor's bytes; returns
    the 32-byte digest as a uint8 device tensor."""
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("commit takes a contiguous device tensor")
    nbytes = t.numel() * t.element_size()
    if digest is None:
        digest = torch.empty(32, dtype=torch.uint8, device=t.device)
    if (not digest.is_cuda or not digest.is_contiguous()
            or digest.numel() * digest.element_size() < 32):
        raise ValueError("digest must be a contiguous device tensor of at least 32 bytes")
    if workspace is None:
        need = commit_workspace(nbytes, chunk_bytes)
        workspace = torch.empty(max(need // 4, 1), dtype=torch.int32, device=t.device)
    wptr, wbytes = _workspace(workspace)
    rc = load().repops_commit(t.data_ptr() if nbytes else None, nbytes, chunk_bytes,
                              digest.data_ptr(), wptr, wbytes, None, _stream(t))
    _check(rc, "repops_commit")
    return digest

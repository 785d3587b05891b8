"""C-ABI checks that need no GPU: the library loads, exports every function
include/repops.h declares, and rejects bad arguments before anything is
launched (every call here fails validation, so no kernel is ever enqueued)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "repops.h")
LIB = os.path.join(ROOT, "paper_2502_19405_amd", "librepops.so")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(repops_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def rp():
    if not os.path.exists(LIB):
        pytest.fail("librepops.so is not built (run python -m paper_2502_19405_amd.build)")
    from paper_2502_19405_amd import repops
    return repops


def test_header_declares_the_operator_calls():
    names = declared_functions()
    for fn in ("repops_matmul", "repops_bmm", "repops_softmax_rows", "repops_layernorm_rows",
               "repops_gelu", "repops_exp", "repops_order_default",
               "repops_softmax_backward_rows", "repops_layernorm_backward_rows",
               "repops_layernorm_backward_workspace", "repops_gelu_backward", "repops_adam_step"):
        assert fn in names


def test_library_exports_every_declared_function(rp):
    lib = ctypes.CDLL(LIB)
    missing = [fn for fn in declared_functions() if not hasattr(lib, fn)]
    assert not missing, missing
    assert set(declared_functions()) == set(rp.EXPORTS)


def test_version_default_order_and_status_strings(rp):
    lib = rp.load()
    assert lib.repops_abi_version() == 2
    o = rp.OrderT()
    lib.repops_order_default(ctypes.byref(o))
    assert (o.version, o.k_block, o.k_inner, o.k_combine, o.row_width, o.row_combine) == (
        1, 64, 0, 0, 64, 0)
    assert list(o.reserved) == [0, 0]
    assert rp.status_str(rp.OK) == "ok"
    assert "order" in rp.status_str(rp.ERR_ORDER)
    assert rp.status_str(99) == "unknown status"


def test_gemm_config_tables(rp):
    tiled = rp.gemm_configs(rp.LAUNCH_GEMM_TILED)
    assert len(tiled) >= 3
    assert all(re.match(r"\d+x\d+x\d+/", n) for n in tiled)
    lib = rp.load()
    assert lib.repops_gemm_config_name(rp.LAUNCH_GEMM_TILED, len(tiled)) is None
    assert lib.repops_gemm_config_count(99) == 0


FAKE_A, FAKE_B, FAKE_C = 0x100000, 0x200000, 0x300000  # never dereferenced

# The calls below pass fake device addresses and must all fail validation.  A
# validation bug would let one reach a kernel launch, so they only run where no
# GPU is present (on a GPU host the launch would read unmapped memory).
no_gpu_only = pytest.mark.skipif(os.path.exists("/dev/kfd"),
                                 reason="fake-pointer validation tests run only without a GPU")


def _order(**kw):
    from paper_2502_19405_amd.repops import Order
    return ctypes.byref(Order(**kw).c())


def _matmul(rp, order=None, m=4, n=4, k=4, A=FAKE_A, lda=4, ta=0, B=FAKE_B, ldb=4, tb=0,
            bias=None, C=FAKE_C, ldc=4, launch=None):
    return rp.load().repops_matmul(order or _order(), m, n, k, A, lda, ta, B, ldb, tb, bias, C,
                                   ldc, launch, None)


@no_gpu_only
def test_matmul_rejections(rp):
    assert _matmul(rp, m=-1) == rp.ERR_SHAPE
    assert _matmul(rp, C=None) == rp.ERR_NULL
    assert _matmul(rp, A=None) == rp.ERR_NULL
    assert _matmul(rp, lda=3) == rp.ERR_STRIDE
    assert _matmul(rp, ldc=3) == rp.ERR_STRIDE
    assert _matmul(rp, ta=2) == rp.ERR_SHAPE
    assert _matmul(rp, C=FAKE_A + 8) == rp.ERR_ALIAS
    assert _matmul(rp, bias=FAKE_C + 4) == rp.ERR_ALIAS
    assert _matmul(rp, order=_order(version=2)) == rp.ERR_ORDER
    assert _matmul(rp, order=_order(k_inner=2)) == rp.ERR_ORDER
    assert _matmul(rp, order=_order(k_combine=1)) == rp.ERR_ORDER
    assert _matmul(rp, order=_order(row_width=48)) == rp.ERR_ORDER
    bad = rp.OrderT()
    rp.load().repops_order_default(ctypes.byref(bad))
    bad.reserved[1] = 1
    assert _matmul(rp, order=ctypes.byref(bad)) == rp.ERR_ORDER
    assert rp.load().repops_matmul(None, 4, 4, 4, FAKE_A, 4, 0, FAKE_B, 4, 0, None, FAKE_C, 4,
                                   None, None) == rp.ERR_ORDER
    # launch descriptors: unknown kind, out-of-table index, block length the tile cannot take
    L = rp.Launch
    assert _matmul(rp, launch=ctypes.byref(L(7).c())) == rp.ERR_LAUNCH
    assert _matmul(rp, launch=ctypes.byref(L(rp.LAUNCH_GEMM_TILED, (99,)).c())) == rp.ERR_LAUNCH
    assert _matmul(rp, launch=ctypes.byref(L(rp.LAUNCH_GEMM_SIMPLE, (1,)).c())) == rp.ERR_LAUNCH
    assert _matmul(rp, order=_order(k_block=24),
                   launch=ctypes.byref(L(rp.LAUNCH_GEMM_TILED, (0,)).c())) == rp.ERR_LAUNCH


@no_gpu_only
def test_bmm_causal_rejections(rp):
    lib = rp.load()
    o = _order()

    def bc(mask=1, lda=8):
        return lib.repops_bmm_causal(o, 1, 1, 8, 8, 8, FAKE_A, 64, 64, lda, 0, FAKE_B, 64, 64, 8,
                                     1, 1.0, FAKE_C, 64, 64, 8, mask, None, None)
    assert bc(mask=0) == rp.ERR_VALUE
    assert bc(mask=3) == rp.ERR_VALUE
    assert bc(lda=7) == rp.ERR_STRIDE
    assert lib.repops_bmm_causal(o, 1, 1, 0, 8, 8, None, 0, 0, 8, 0, None, 0, 0, 8, 0, 1.0, None,
                                 0, 0, 8, 2, None, None) == rp.OK


@no_gpu_only
def test_matmul_grouped_rejections(rp):
    lib = rp.load()
    o = _order()
    D = rp.GemmDescT

    def desc(m=8, n=8, k=8, A=FAKE_A, lda=8, ta=0, B=FAKE_B, ldb=8, tb=0, bias=None, C=FAKE_C,
             ldc=8):
        return D(m, n, k, A, lda, ta, B, ldb, tb, bias, C, ldc)

    def call(*ds, count=None, order=None, launch=None):
        arr = (D * max(len(ds), 1))(*ds)
        return lib.repops_matmul_grouped(order or o, len(ds) if count is None else count, arr,
                                         launch, None)
    assert lib.repops_matmul_grouped(o, 0, None, None, None) == rp.OK
    assert lib.repops_matmul_grouped(o, 2, None, None, None) == rp.ERR_NULL
    assert call(desc(), count=-1) == rp.ERR_SHAPE
    assert call(*[desc(C=FAKE_C + 0x1000 * i) for i in range(9)]) == rp.ERR_SHAPE
    assert call(desc(), order=_order(version=0)) == rp.ERR_ORDER
    assert call(desc(), launch=ctypes.byref(rp.Launch(rp.LAUNCH_GEMM_MFMA, (0,)).c())) == \
        rp.ERR_LAUNCH
    assert call(desc(ldc=7)) == rp.ERR_STRIDE
    assert call(desc(C=FAKE_A + 4)) == rp.ERR_ALIAS                  # over its own A
    assert call(desc(), desc(C=FAKE_C + 16)) == rp.ERR_ALIAS         # two outputs overlap
    assert call(desc(), desc(A=FAKE_C + 8, C=FAKE_D)) == rp.ERR_ALIAS  # reads another's output
    assert call(desc(), desc(bias=FAKE_C + 4, C=FAKE_D)) == rp.ERR_ALIAS
    assert call(desc(m=0), desc(n=0, C=FAKE_D)) == rp.OK               # nothing to compute


@no_gpu_only
def test_matmul_gelu_rejections(rp):
    lib = rp.load()
    FAKE_G = 0x500000

    def call(order=None, m=4, n=4, k=4, A=FAKE_A, lda=4, ta=0, B=FAKE_B, ldb=4, tb=0, bias=None,
             H=FAKE_C, ldh=4, G=FAKE_G, ldg=4, launch=None):
        return lib.repops_matmul_gelu(order or _order(), m, n, k, A, lda, ta, B, ldb, tb, bias, H,
                                      ldh, G, ldg, launch, None)
    assert call(order=_order(version=2)) == rp.ERR_ORDER
    assert call(m=-1) == rp.ERR_SHAPE
    assert call(H=None) == rp.ERR_NULL
    assert call(G=None) == rp.ERR_NULL
    assert call(ldh=3) == rp.ERR_STRIDE
    assert call(ldg=3) == rp.ERR_STRIDE
    assert call(H=FAKE_A + 8) == rp.ERR_ALIAS            # H over A (the matmul checks)
    assert call(G=FAKE_C + 4) == rp.ERR_ALIAS            # G over H
    assert call(G=FAKE_A + 60) == rp.ERR_ALIAS           # G over A's last element
    assert call(G=FAKE_B) == rp.ERR_ALIAS                # G over B
    assert call(bias=FAKE_G + 12) == rp.ERR_ALIAS        # bias inside G
    assert call(launch=ctypes.byref(rp.Launch(7).c())) == rp.ERR_LAUNCH
    # nothing to write: succeeds without touching any pointer or the device
    assert call(m=0, A=None, B=None, H=None, G=None) == rp.OK


@no_gpu_only
def test_matmul_gelu_backward_rejections(rp):
    lib = rp.load()
    FAKE_X = 0x500000

    def call(order=None, m=4, n=4, k=4, A=FAKE_A, lda=4, ta=0, B=FAKE_B, ldb=4, tb=0, X=FAKE_X,
             ldx=4, C=FAKE_C, ldc=4, launch=None):
        return lib.repops_matmul_gelu_backward(order or _order(), m, n, k, A, lda, ta, B, ldb, tb,
                                               X, ldx, C, ldc, launch, None)
    assert call(order=_order(version=2)) == rp.ERR_ORDER
    assert call(m=-1) == rp.ERR_SHAPE
    assert call(C=None) == rp.ERR_NULL
    assert call(X=None) == rp.ERR_NULL
    assert call(ldx=3) == rp.ERR_STRIDE
    assert call(C=FAKE_X + 8) == rp.ERR_ALIAS            # C over X
    assert call(C=FAKE_B + 60) == rp.ERR_ALIAS           # C over B (the matmul checks)
    assert call(launch=ctypes.byref(rp.Launch(7).c())) == rp.ERR_LAUNCH
    assert call(m=0, A=None, B=None, X=None, C=None) == rp.OK
    # the grouped form: gelu_in per product
    D = rp.GemmDescT

    def desc(bias=None, C=FAKE_C, gelu_in=FAKE_X, ld_gelu_in=8):
        return D(8, 8, 8, FAKE_A, 8, 0, FAKE_B, 8, 0, bias, C, 8, gelu_in, ld_gelu_in)

    def grouped(*ds):
        arr = (D * len(ds))(*ds)
        return lib.repops_matmul_grouped(_order(), len(ds), arr, None, None)
    assert grouped(desc(ld_gelu_in=7)) == rp.ERR_STRIDE
    assert grouped(desc(bias=0x600000)) == rp.ERR_VALUE          # no bias with gelu_in
    assert grouped(desc(C=FAKE_X + 16)) == rp.ERR_ALIAS          # C over its own gelu_in
    assert grouped(desc(), desc(C=FAKE_X + 16, gelu_in=None)) == rp.ERR_ALIAS  # over another's


def test_matmul_zero_sized_is_a_noop(rp):
    # nothing to write: succeeds without touching any pointer or the device
    assert _matmul(rp, m=0, A=None, B=None, C=None) == rp.OK
    assert _matmul(rp, n=0, A=None, B=None, C=None) == rp.OK


@no_gpu_only
def test_bmm_rejections(rp):
    lib = rp.load()

    def call(**kw):
        args = dict(b0=2, b1=3, m=4, n=4, k=4, A=FAKE_A, sa0=48, sa1=16, lda=4, ta=0, B=FAKE_B,
                    sb0=48, sb1=16, ldb=4, tb=0, alpha=1.0, C=FAKE_C, sc0=48, sc1=16, ldc=4)
        args.update(kw)
        return lib.repops_bmm(_order(), *args.values(), None, None)

    assert call(b0=-1) == rp.ERR_SHAPE
    # A spans elements [0, 48 + 2*16 + 3*4 + 4) = [0, 96): C starting at 90 overlaps it
    assert call(C=FAKE_A + 4 * 90) == rp.ERR_ALIAS
    assert call(ldb=3) == rp.ERR_STRIDE
    assert call(b1=0, A=None, B=None, C=None) == rp.OK
    # no two output elements may share an address: batch strides 0 or shorter
    # than a batch element's span are rejected...
    assert call(sc1=0) == rp.ERR_STRIDE
    assert call(sc1=15) == rp.ERR_STRIDE      # a 4 x 4 element with ldc 4 spans 16
    assert call(sc0=40) == rp.ERR_STRIDE      # b1 = 3 elements of 16 span 48
    assert call(sc0=-16, sc1=16) == rp.ERR_STRIDE
    # ...while interleaved dense layouts pass that check and reach the alias
    # check after it: heads within rows ([b0][m][b1][n]: sc0 48, sc1 4, ldc 12)
    # and batch dimensions in either order
    for sc0, sc1, ldc in ((48, 4, 12), (16, 32, 4), (4, 96, 12)):
        assert call(sc0=sc0, sc1=sc1, ldc=ldc, C=FAKE_A + 4 * 8) == rp.ERR_ALIAS, (sc0, sc1, ldc)
    assert call(sc0=48, sc1=3, ldc=12, C=FAKE_A + 4 * 8) == rp.ERR_STRIDE


@no_gpu_only
def test_rows_and_elementwise_rejections(rp):
    lib = rp.load()
    o = _order()
    assert lib.repops_softmax_rows(o, 4, 8, FAKE_A, 7, FAKE_C, 8, 0, None, None) == rp.ERR_STRIDE
    assert lib.repops_softmax_rows(o, 4, 8, FAKE_A, 8, FAKE_A + 4, 8, 0, None, None) == rp.ERR_ALIAS
    assert lib.repops_softmax_rows(o, 4, 8, FAKE_A, 8, FAKE_C, 8, -1, None, None) == rp.ERR_SHAPE
    assert lib.repops_softmax_rows(o, 0, 8, None, 8, None, 8, 0, None, None) == rp.OK
    wave = ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (3,)).c())
    assert lib.repops_softmax_rows(o, 4, 8, FAKE_A, 8, FAKE_C, 8, 0, wave, None) == rp.ERR_LAUNCH
    wave4 = ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (4,)).c())
    assert lib.repops_softmax_rows(_order(row_width=32), 4, 8, FAKE_A, 8, FAKE_C, 8, 0, wave4,
                                   None) == rp.ERR_LAUNCH
    # split rows (ROWS_WAVE p[1] = waves per row): 2, 4 or 8, one row per block, and a
    # row of at most 32 values per lane
    for p in ((1, 3), (1, 16), (1, 32), (2, 4), (4, 2)):
        bad = ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, p).c())
        assert lib.repops_softmax_rows(o, 4, 8, FAKE_A, 8, FAKE_C, 8, 0, bad, None) == \
            rp.ERR_LAUNCH, p
    wide = ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (1, 2)).c())
    assert lib.repops_softmax_rows(o, 4, 4097, FAKE_A, 4097, FAKE_C, 4097, 0, wide, None) == \
        rp.ERR_LAUNCH
    assert lib.repops_softmax_rows(_order(row_width=32), 4, 8, FAKE_A, 8, FAKE_C, 8, 0, wide,
                                   None) == rp.ERR_LAUNCH
    assert lib.repops_layernorm_rows(o, 4, 8, FAKE_A, 8, None, None, 1e-5, FAKE_C, 8, None, None,
                                     ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (1, 5)).c()),
                                     None) == rp.ERR_LAUNCH
    # the backward row operations take splits too, under the same rules
    assert lib.repops_softmax_backward_rows(o, 4, 4097, FAKE_A, 4097, FAKE_B, 4097, FAKE_C, 4097,
                                            0, wide, None) == rp.ERR_LAUNCH
    assert lib.repops_layernorm_rows(o, 4, 0, FAKE_A, 8, None, None, 1e-5, FAKE_C, 8, None, None,
                                     None, None) == rp.ERR_SHAPE
    assert lib.repops_layernorm_rows(o, 4, 8, FAKE_A, 8, FAKE_C + 4, None, 1e-5, FAKE_C, 8, None,
                                     None, None, None) == rp.ERR_ALIAS
    # the row statistics may touch no input, not Y and not each other (X and Y
    # are 4 x 8 floats, gamma 8 floats, each statistic 4 floats)
    for gamma, mean, rstd in ((None, FAKE_A + 8, None),        # inside X
                              (None, None, FAKE_C + 64),       # inside Y
                              (None, FAKE_B, FAKE_B + 8),      # mean and rstd overlap
                              (FAKE_B, FAKE_B + 16, None)):    # inside gamma
        assert lib.repops_layernorm_rows(o, 4, 8, FAKE_A, 8, gamma, None, 1e-5, FAKE_C, 8, mean,
                                         rstd, None, None) == rp.ERR_ALIAS, (gamma, mean, rstd)
    assert lib.repops_gelu(o, -1, FAKE_A, FAKE_C, None, None) == rp.ERR_SHAPE
    assert lib.repops_gelu(o, 8, FAKE_A, FAKE_A + 4, None, None) == rp.ERR_ALIAS
    assert lib.repops_exp(o, 8, None, FAKE_C, None, None) == rp.ERR_NULL
    ew = ctypes.byref(rp.Launch(rp.LAUNCH_ELEMENTWISE, (100,)).c())
    assert lib.repops_exp(o, 8, FAKE_A, FAKE_C, ew, None) == rp.ERR_LAUNCH
    assert lib.repops_exp(o, 0, None, None, None, None) == rp.OK


FAKE_D, FAKE_M, FAKE_R, FAKE_G, FAKE_W = 0x400000, 0x500000, 0x600000, 0x700000, 0x800000


@no_gpu_only
def test_training_rejections(rp):
    lib = rp.load()
    o = _order()
    sbw = lib.repops_softmax_backward_rows
    assert sbw(o, 4, 8, FAKE_A, 8, FAKE_B, 8, FAKE_C, 7, 0, None, None) == rp.ERR_STRIDE
    assert sbw(o, 4, 8, FAKE_A, 8, None, 8, FAKE_C, 8, 0, None, None) == rp.ERR_NULL
    assert sbw(o, 4, 8, FAKE_A, 8, FAKE_B, 8, FAKE_A + 4, 8, 0, None, None) == rp.ERR_ALIAS
    assert sbw(o, 4, 8, FAKE_A, 8, FAKE_B, 8, FAKE_B, 9, 0, None, None) == rp.ERR_ALIAS
    assert sbw(o, 4, 8, FAKE_A, 8, FAKE_B, 8, FAKE_C, 8, -1, None, None) == rp.ERR_SHAPE
    assert sbw(o, 0, 8, None, 8, None, 8, None, 8, 0, None, None) == rp.OK

    ws = ctypes.c_uint64(1)
    assert lib.repops_layernorm_backward_workspace(o, 4096, 768, ctypes.byref(ws)) == rp.OK
    assert ws.value == 2 * 64 * 768 * 4
    assert lib.repops_layernorm_backward_workspace(o, 64, 768, ctypes.byref(ws)) == rp.OK
    assert ws.value == 0
    assert lib.repops_layernorm_backward_workspace(_order(k_block=0), 4096, 768,
                                                   ctypes.byref(ws)) == rp.OK
    assert ws.value == 0
    assert lib.repops_layernorm_backward_workspace(o, 64, 768, None) == rp.ERR_NULL

    def lnb(rows=128, cols=8, X=FAKE_A, ldx=8, dY=FAKE_B, lddy=8, mean=FAKE_M, rstd=FAKE_R,
            gamma=None, dX=FAKE_C, lddx=8, dg=FAKE_D, db=FAKE_D + 64, ws=FAKE_W, wsb=1 << 20,
            order=None):
        return lib.repops_layernorm_backward_rows(order or o, rows, cols, X, ldx, dY, lddy, mean,
                                                  rstd, gamma, dX, lddx, dg, db, ws, wsb, None,
                                                  None)
    assert lnb(cols=0) == rp.ERR_SHAPE
    assert lnb(ws=None) == rp.ERR_WORKSPACE
    assert lnb(wsb=2 * 2 * 8 * 4 - 4) == rp.ERR_WORKSPACE
    assert lnb(mean=None) == rp.ERR_NULL
    assert lnb(lddx=7) == rp.ERR_STRIDE
    assert lnb(dX=FAKE_A + 4) == rp.ERR_ALIAS           # dX partly over X
    assert lnb(db=FAKE_D + 16) == rp.ERR_ALIAS          # dgamma and dbeta overlap
    assert lnb(ws=FAKE_D) == rp.ERR_ALIAS               # workspace over dgamma
    assert lnb(dg=FAKE_M) == rp.ERR_ALIAS               # dgamma over mean
    assert lnb(gamma=FAKE_C + 8) == rp.ERR_ALIAS        # gamma inside dX
    assert lnb(order=_order(version=0)) == rp.ERR_ORDER
    assert lnb(rows=4, cols=0, dX=None, dg=None, db=None) == rp.ERR_SHAPE
    assert lnb(rows=0, cols=0) == rp.OK

    assert lib.repops_gelu_backward(o, 8, FAKE_A, FAKE_B, FAKE_A + 4, None, None) == rp.ERR_ALIAS
    assert lib.repops_gelu_backward(o, 8, FAKE_A, FAKE_B, FAKE_B + 4, None, None) == rp.ERR_ALIAS
    assert lib.repops_gelu_backward(o, 8, FAKE_A, None, FAKE_C, None, None) == rp.ERR_NULL
    assert lib.repops_gelu_backward(o, -1, FAKE_A, FAKE_B, FAKE_C, None, None) == rp.ERR_SHAPE

    def adam(n=8, p=FAKE_A, g=FAKE_B, m=FAKE_C, v=FAKE_D, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8,
             wd=0.0, step=1, dec=1):
        return lib.repops_adam_step(o, n, p, g, m, v, lr, b1, b2, eps, wd, step, dec, None, None)
    assert adam(step=0) == rp.ERR_VALUE
    assert adam(b1=1.0) == rp.ERR_VALUE
    assert adam(b2=-0.1) == rp.ERR_VALUE
    assert adam(lr=float("inf")) == rp.ERR_VALUE
    assert adam(eps=float("nan")) == rp.ERR_VALUE
    assert adam(dec=2) == rp.ERR_VALUE
    assert adam(m=None) == rp.ERR_NULL
    assert adam(m=FAKE_A + 16) == rp.ERR_ALIAS
    assert adam(v=FAKE_C) == rp.ERR_ALIAS
    assert adam(n=-1) == rp.ERR_SHAPE
    assert adam(n=0, p=None, g=None, m=None, v=None) == rp.OK
    assert rp.status_str(rp.ERR_WORKSPACE).startswith("workspace")

    # the no-allocation LayerNorm backward: its fixed scratch bounds the size
    def nb(rows=64, cols=8, mean=FAKE_M, order=None, dg=FAKE_D):
        return lib.repops_layernorm_backward_rows_noalloc(
            order or o, rows, cols, FAKE_A, cols, FAKE_B, cols, mean, FAKE_R, None, FAKE_C, cols,
            dg, None, None, None)
    assert rp.NOALLOC_SCRATCH_BYTES == 8 << 20
    assert nb(rows=262144, cols=768) == rp.ERR_SCRATCH     # 2 * 4096 * 768 * 4 B > 8 MiB
    assert nb(rows=64 * 1366, cols=768) == rp.ERR_SCRATCH  # just over: 1366 blocks
    assert nb(rows=64, mean=None) == rp.ERR_NULL           # one block: no scratch needed
    assert nb(rows=64, dg=FAKE_C + 4) == rp.ERR_ALIAS
    assert nb(cols=0) == rp.ERR_SHAPE
    assert nb(order=_order(version=0)) == rp.ERR_ORDER
    assert nb(rows=0, cols=8, dg=None) == rp.OK
    assert "scratch" in rp.status_str(rp.ERR_SCRATCH)


@no_gpu_only
def test_llama_rejections(rp):
    lib = rp.load()
    o = _order()
    assert lib.repops_sincos(o, 8, FAKE_A, None, None, None, None) == rp.ERR_NULL
    assert lib.repops_sincos(o, 8, FAKE_A, FAKE_B, FAKE_B + 4, None, None) == rp.ERR_ALIAS
    assert lib.repops_sincos(o, 8, FAKE_A, FAKE_A, FAKE_C, None, None) == rp.ERR_ALIAS
    assert lib.repops_sincos(o, -1, FAKE_A, FAKE_B, None, None, None) == rp.ERR_SHAPE

    def rope(rows=4, heads=2, hd=8, X=FAKE_A, ldx=16, inv=FAKE_D, period=0, offset=0, inverse=0,
             Y=FAKE_C, ldy=16, launch=None):
        return lib.repops_rope(o, rows, heads, hd, X, ldx, inv, period, offset, inverse, Y, ldy,
                               launch, None)
    assert rope(hd=7) == rp.ERR_SHAPE
    assert rope(ldx=15) == rp.ERR_STRIDE
    assert rope(inv=None) == rp.ERR_NULL
    assert rope(Y=FAKE_A + 4) == rp.ERR_ALIAS
    assert rope(inv=FAKE_C + 8) == rp.ERR_ALIAS
    assert rope(inverse=2) == rp.ERR_VALUE
    assert rope(offset=1 << 24) == rp.ERR_SHAPE
    assert rope(period=-1) == rp.ERR_SHAPE
    assert rope(launch=ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (3,)).c())) == rp.ERR_LAUNCH
    # no split kernel for the rotary embedding
    assert rope(launch=ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (1, 2)).c())) == rp.ERR_LAUNCH
    assert rope(launch=ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_GENERIC).c())) == rp.ERR_LAUNCH
    assert rope(rows=0, X=None, Y=None, inv=None) == rp.OK

    rms = lib.repops_rmsnorm_rows
    assert rms(o, 4, 0, FAKE_A, 8, None, 1e-5, FAKE_C, 8, None, None, None) == rp.ERR_SHAPE
    assert rms(o, 4, 8, FAKE_A, 8, FAKE_C + 4, 1e-5, FAKE_C, 8, None, None, None) == rp.ERR_ALIAS
    assert rms(o, 4, 8, FAKE_A, 8, None, 1e-5, FAKE_C, 8, FAKE_A + 8, None, None) == rp.ERR_ALIAS
    ws = ctypes.c_uint64(0)
    assert lib.repops_rmsnorm_backward_workspace(o, 4096, 4096, ctypes.byref(ws)) == rp.OK
    assert ws.value == 2 * 64 * 4096 * 4
    rb = lib.repops_rmsnorm_backward_rows
    assert rb(o, 128, 8, FAKE_A, 8, FAKE_B, 8, None, None, FAKE_C, 8, FAKE_D, FAKE_W, 1 << 20,
              None, None) == rp.ERR_NULL
    assert rb(o, 128, 8, FAKE_A, 8, FAKE_B, 8, FAKE_R, None, FAKE_C, 8, FAKE_D, None, 0,
              None, None) == rp.ERR_WORKSPACE
    assert rb(o, 128, 8, FAKE_A, 8, FAKE_B, 8, FAKE_R, None, FAKE_C, 8, FAKE_R, FAKE_W, 1 << 20,
              None, None) == rp.ERR_ALIAS

    assert lib.repops_silu(o, 8, FAKE_A, FAKE_A + 4, None, None) == rp.ERR_ALIAS
    assert lib.repops_swiglu(o, 8, FAKE_A, None, FAKE_C, None, None) == rp.ERR_NULL
    assert lib.repops_swiglu(o, 8, FAKE_A, FAKE_B, FAKE_B + 4, None, None) == rp.ERR_ALIAS
    sb = lib.repops_swiglu_backward
    assert sb(o, 8, FAKE_A, FAKE_B, FAKE_D, FAKE_C, FAKE_C + 4, None, None) == rp.ERR_ALIAS
    assert sb(o, 8, FAKE_A, FAKE_B, FAKE_D, FAKE_A + 4, FAKE_C, None, None) == rp.ERR_ALIAS
    assert sb(o, 8, FAKE_A, FAKE_B, None, FAKE_C, FAKE_W, None, None) == rp.ERR_NULL
    assert sb(o, 0, None, None, None, None, None, None, None) == rp.OK


@no_gpu_only
def test_commit_rejections(rp):
    lib = rp.load()
    n = ctypes.c_uint64(0)
    assert lib.repops_commit_workspace(1 << 20, 1024, ctypes.byref(n)) == rp.OK
    assert n.value == 32 * (1024 + 512)
    assert lib.repops_commit_workspace(0, 1024, ctypes.byref(n)) == rp.OK and n.value == 0
    assert lib.repops_commit_workspace(10, 0, ctypes.byref(n)) == rp.ERR_SHAPE
    assert lib.repops_commit_workspace(10, 64, None) == rp.ERR_NULL
    c = lib.repops_commit
    assert c(FAKE_A, 4096, 1024, None, FAKE_W, 1 << 20, None, None) == rp.ERR_NULL
    assert c(None, 4096, 1024, FAKE_C, FAKE_W, 1 << 20, None, None) == rp.ERR_NULL
    assert c(FAKE_A, 4096, 1024, FAKE_C, None, 0, None, None) == rp.ERR_WORKSPACE
    assert c(FAKE_A, 4096, 1024, FAKE_C, FAKE_W, 32 * 6 - 1, None, None) == rp.ERR_WORKSPACE
    assert c(FAKE_A, 4096, 1024, FAKE_A + 100, FAKE_W, 1 << 20, None, None) == rp.ERR_ALIAS
    assert c(FAKE_A, 4096, 1024, FAKE_C, FAKE_A + 64, 1 << 20, None, None) == rp.ERR_ALIAS
    assert c(FAKE_A, 4096, 1024, FAKE_C, FAKE_W + 2, 1 << 20, None, None) == rp.ERR_STRIDE
    wave = ctypes.byref(rp.Launch(rp.LAUNCH_ROWS_WAVE, (4,)).c())
    assert c(FAKE_A, 4096, 1024, FAKE_C, FAKE_W, 1 << 20, wave, None) == rp.ERR_LAUNCH


def test_binding_passes_row_strides_and_checks_output_shapes(rp):
    # the binding hands the library a tensor's own row stride (rows that
    # overlap, as in an expanded view, are then rejected there, not widened),
    # and every output must have exactly the shape the call writes: both
    # checks run before any pointer is taken, so host tensors show them here
    import torch
    X = torch.zeros(4, 8)
    assert rp._rows(X, "X") == (4, 8, 8)
    assert rp._rows(torch.zeros(8).expand(4, 8), "X") == (4, 8, 0)
    assert rp._rows(torch.zeros(40)[:8].view(1, 8), "X") == (1, 8, 8)
    assert rp._rows(torch.zeros(4, 12)[:, 2:10], "X") == (4, 8, 12)
    with pytest.raises(ValueError, match="unit column stride"):
        rp._rows(torch.zeros(8, 4).t(), "X")
    assert rp._rows_as(torch.zeros(4, 12)[:, :8], 4, 8, "out") == 12
    with pytest.raises(ValueError, match=r"must be \[4, 8\]"):
        rp._rows_as(torch.zeros(3, 8), 4, 8, "out")
    short, narrow = torch.zeros(3, 8), torch.zeros(4, 7)
    for bad in (short, narrow):
        for call in (lambda: rp.softmax_rows(X, out=bad),
                     lambda: rp.layernorm_rows(X, out=bad),
                     lambda: rp.rmsnorm_rows(X, out=bad),
                     lambda: rp.softmax_backward_rows(X, X, out=bad)):
            with pytest.raises(ValueError):
                call()
    with pytest.raises(ValueError, match="rows"):
        rp.rope(X, 2, 4, torch.zeros(2), out=short)
    with pytest.raises(ValueError, match="out must be"):
        rp.bmm(torch.zeros(2, 3, 4, 5), torch.zeros(2, 3, 5, 6), out=torch.zeros(1, 3, 4, 6))
    # a caller's workspace must be device memory the library may fill contiguously
    with pytest.raises(ValueError, match="workspace"):
        rp._workspace(torch.zeros(16))


def test_binding_fails_loudly_without_library(tmp_path):
    from paper_2502_19405_amd import repops
    with pytest.raises(RuntimeError, match="not found"):
        repops.load(str(tmp_path / "missing.so"))

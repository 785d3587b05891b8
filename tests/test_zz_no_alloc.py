"""The no-allocation LayerNorm backward (repops_layernorm_backward_rows_noalloc)
against the workspace entry point (repops_layernorm_backward_rows) and the
oracle, bit for bit: two calls in a row, the second smaller than the first
(the fixed scratch array keeps the first call's partials), then a call of one
row block (no scratch) and a call past the scratch limit (refused, nothing
enqueued).  Every call goes through the C ABI, with the caller's outputs
passed in, and torch's allocator must not grow during the no-allocation
calls."""
import numpy as np
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


def ln_inputs(seed, rows, cols):
    g = inputs.rng(seed)
    X = inputs.normal(g, (rows, cols), var=0.5)
    gamma = (1 + inputs.uniform(g, (cols,), -0.1, 0.1)).astype(np.float32)
    beta = inputs.uniform(g, (cols,), -0.1, 0.1)
    _, mean, rstd = oracle.layernorm_rows(X, gamma, beta, with_stats=True)
    dY = inputs.normal(g, (rows, cols), var=1e-2)
    return X, dY, mean, rstd, gamma


def run_both(rp, case, launch=None):
    import torch
    X, dY, mean, rstd, gamma = (dev(a) for a in case)
    rows, cols = X.shape
    # the workspace entry point, workspace allocated by the binding
    ref = rp.layernorm_backward_rows(X, dY, mean, rstd, gamma, launch=launch)
    outs = (torch.full((rows, cols), float("nan"), device="cuda:0"),
            torch.full((cols,), float("nan"), device="cuda:0"),
            torch.full((cols,), float("nan"), device="cuda:0"))
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    got = rp.layernorm_backward_rows_noalloc(X, dY, mean, rstd, gamma, *outs, launch=launch)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    return [host(t) for t in ref], [host(t) for t in got]


@pytest.mark.parametrize("launch_name", ["auto", "wave8", "generic"])
def test_noalloc_equals_workspace_entry_two_calls_second_smaller(rp, launch_name):
    launch = {"auto": None, "wave8": rp.Launch(rp.LAUNCH_ROWS_WAVE, (8,)),
              "generic": rp.Launch(rp.LAUNCH_ROWS_GENERIC)}[launch_name]
    # 4096 x 768: 64 row blocks (column-split kernels under auto); then
    # 1000 x 300: 16 blocks, a ragged last block; then 64 x 768: one block
    for seed, rows, cols in ((1, 4096, 768), (2, 1000, 300), (3, 64, 768)):
        announce("noalloc layernorm backward", launch_name, rows, cols)
        case = ln_inputs(seed, rows, cols)
        ref, got = run_both(rp, case, launch)
        want = oracle.layernorm_backward_rows(*case)
        for r, g, w, what in zip(ref, got, want, ("dX", "dgamma", "dbeta")):
            assert_bits_equal(g, r, f"{what} noalloc vs workspace entry {rows}x{cols}")
            assert_bits_equal(g, w, f"{what} noalloc vs oracle {rows}x{cols}")


def test_noalloc_largest_scratch_then_small(rp):
    """65536 x 768 fills 6 MiB of the 8 MiB scratch (1024 row blocks); the next
    call is a small one."""
    for seed, rows, cols in ((4, 65536, 768), (5, 200, 96)):
        announce("noalloc layernorm backward", rows, cols)
        case = ln_inputs(seed, rows, cols)
        ref, got = run_both(rp, case)
        for r, g, what in zip(ref, got, ("dX", "dgamma", "dbeta")):
            assert_bits_equal(g, r, f"{what} noalloc vs workspace entry {rows}x{cols}")


def test_noalloc_refuses_past_its_scratch(rp):
    import torch
    rows, cols = 262144, 768  # 4096 row blocks: 25 MB of partials
    X = torch.zeros((1, cols), device="cuda:0").expand(rows, cols)
    v = torch.zeros(rows, device="cuda:0")
    p = torch.zeros(cols, device="cuda:0")
    with pytest.raises(rp.RepopsError) as e:
        rp.layernorm_backward_rows_noalloc(X, X, v, v, None, None, p, None)
    assert e.value.code == rp.ERR_SCRATCH

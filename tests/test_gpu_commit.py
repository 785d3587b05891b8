"""GPU parity of the tensor commitment (repops_commit) against the CPU oracle:
byte-identical 32-byte digests for every size class (empty, one byte, one
chunk, chunk +- 1, odd and power-of-two leaf counts, trees deeper than the
single-workgroup top), unaligned data and chunk sizes off the vector path, and
model-sized tensors."""
import numpy as np
import pytest

import oracle
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


def gpu_commit(rp, buf_u8, chunk):
    """Digest of a uint8 host buffer, placed at the start of a device tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(buf_u8)).to("cuda:0")
    return bytes(host(rp.commit(t, chunk)).tobytes())


@pytest.mark.parametrize("chunk", [64, 1024, 4096, 100])
def test_commit_sizes(rp, chunk):
    g = inputs.rng(950 + chunk)
    # leaf counts around the 256 leaves one workgroup reduces, and (64-byte
    # chunks) more than 512 x 256 leaves, so a level launch runs as well
    sizes = [0, 1, 3, 63, 64, 65, chunk - 1, chunk, chunk + 1, 2 * chunk, 3 * chunk + 7,
             255 * chunk, 256 * chunk, 257 * chunk + 5, 513 * chunk, 512 * chunk,
             1025 * chunk - 3, 5000 * chunk + 1]
    if chunk == 64:
        sizes.append((512 * 256 + 300) * chunk + 9)
    for n in sizes:
        if n < 0:
            continue
        data = g.integers(0, 256, n).astype(np.uint8)
        announce("commit", chunk, n)
        assert gpu_commit(rp, data, chunk) == oracle.commit(data, chunk), (chunk, n)


def test_commit_unaligned_views(rp):
    import torch
    g = inputs.rng(951)
    data = g.integers(0, 256, 70001).astype(np.uint8)
    base = torch.from_numpy(data).to("cuda:0")
    for off in (1, 2, 3, 4, 8, 12, 16):
        announce("commit unaligned", off)
        view = base[off:]
        got = bytes(host(rp.commit(view, 1024)).tobytes())
        assert got == oracle.commit(data[off:], 1024), off


def test_commit_float_tensors(rp):
    g = inputs.rng(952)
    for shape in ((768, 3072), (4096, 768), (1000, 999)):
        X = inputs.normal(g, shape)
        announce("commit tensor", shape)
        got = bytes(host(rp.commit(dev(X), 1024)).tobytes())
        assert got == oracle.commit(X, 1024), shape


def test_commit_llama_mlp_weight(rp):
    """A Llama-8B feed-forward weight, 4096 x 14336 fp32 (235 MB, 229376
    leaves, 18 tree levels)."""
    g = inputs.rng(953)
    W = inputs.normal(g, (4096, 14336), var=4e-4)
    announce("commit llama weight")
    got = bytes(host(rp.commit(dev(W), 1024)).tobytes())
    assert got == oracle.commit(W, 1024)

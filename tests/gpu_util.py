"""Helpers for the GPU parity tests: device transfer, bitwise comparison of
device results, and a flushed progress line before every GPU step."""
import sys

import numpy as np


def announce(*parts):
    print("[gpu-step]", *parts, flush=True)
    sys.stdout.flush()


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().to("cpu").numpy()


def same_bits(a, b):
    """Bitwise equality of two device float32 tensors (on the device)."""
    import torch
    return bool(torch.equal(a.contiguous().view(torch.int32), b.contiguous().view(torch.int32)))

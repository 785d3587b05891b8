"""Pins for the oracle's tensor commitments (no GPU): SHA-256 against the
standard's example digests, its constants against their definitions, and an
independent implementation (Python's hashlib) on every message length through
several blocks; the Merkle commitment against an independent recursive
statement of RFC 6962's Merkle Tree Hash built on hashlib, and the level-wise
pairing with odd-node promotion (the GPU's schedule) against the same."""
import hashlib
import json
import os
import re

import numpy as np
import pytest

import oracle
from paper_2502_19405_amd import inputs

HERE = os.path.dirname(os.path.abspath(__file__))


def test_sha256_standard_examples(ref):
    spec = json.load(open(os.path.join(HERE, "golden", "sha256_vectors.json")))
    for v in spec["vectors"]:
        msg = v["message_ascii"].encode() * v["repeat"]
        assert oracle.sha256(msg, lib=ref).hex() == v["sha256"], v["message_ascii"][:8]


def check_sha_constants(src):
    """Round constants: first 32 bits of the fractional parts of the cube roots
    of the first 64 primes; initial hash: of the square roots of the first 8
    primes (FIPS 180-4, Sections 4.2.2 and 5.3.3) -- exact integer roots."""
    primes = [p for p in range(2, 320) if all(p % q for q in range(2, int(p ** 0.5) + 1))][:64]

    def frac_bits(p, root):
        # floor(frac(p^(1/root)) * 2^32) via the integer root of p * 2^(32*root)
        n = p << (32 * root)
        lo, hi = 0, 1 << (32 + 10)
        while lo < hi:  # largest x with x^root <= n
            mid = (lo + hi + 1) // 2
            if mid ** root <= n:
                lo = mid
            else:
                hi = mid - 1
        return lo & 0xFFFFFFFF

    def table(name):
        body = re.search(name + r"\[\d+\] = \{(.*?)\};", src, re.S).group(1)
        return [int(t.strip().rstrip("u"), 16) for t in body.split(",") if t.strip()]

    assert table("SHA_K") == [frac_bits(p, 3) for p in primes]
    assert table("SHA_H0") == [frac_bits(p, 2) for p in primes[:8]]


def test_sha256_constants_match_definitions():
    check_sha_constants(open(os.path.join(os.path.dirname(oracle.__file__), "repops_ref.c")).read())


def test_sha256_every_length_against_hashlib(ref):
    g = inputs.rng(900)
    for n in list(range(0, 300)) + [1000, 4095, 4096, 4097, 100000]:
        m = g.integers(0, 256, n).astype(np.uint8).tobytes()
        assert oracle.sha256(m, lib=ref) == hashlib.sha256(m).digest(), n


def mth_recursive(data: bytes, chunk: int) -> bytes:
    """RFC 6962, Section 2.1, stated recursively with hashlib."""
    leaves = [data[i:i + chunk] for i in range(0, len(data), chunk)]

    def mth(d):
        if len(d) == 0:
            return hashlib.sha256(b"").digest()
        if len(d) == 1:
            return hashlib.sha256(b"\x00" + d[0]).digest()
        k = 1
        while 2 * k < len(d):
            k *= 2
        return hashlib.sha256(b"\x01" + mth(d[:k]) + mth(d[k:])).digest()

    return mth(leaves)


def mth_levels(data: bytes, chunk: int) -> bytes:
    """Level by level: adjacent pairs hashed, an odd last node carried up."""
    if not data:
        return hashlib.sha256(b"").digest()
    level = [hashlib.sha256(b"\x00" + data[i:i + chunk]).digest()
             for i in range(0, len(data), chunk)]
    while len(level) > 1:
        nxt = [hashlib.sha256(b"\x01" + level[i] + level[i + 1]).digest()
               for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


@pytest.mark.parametrize("chunk", [64, 1024, 4096])
def test_commit_against_rfc6962(ref, chunk):
    g = inputs.rng(901 + chunk)
    sizes = [0, 1, 3, chunk - 1, chunk, chunk + 1, 2 * chunk, 3 * chunk - 5, 5 * chunk, 7 * chunk + 1,
             8 * chunk, 9 * chunk, 33 * chunk + 17, 100 * chunk]
    for n in sizes:
        data = g.integers(0, 256, n).astype(np.uint8).tobytes()
        want = mth_recursive(data, chunk)
        assert oracle.commit(data, chunk, lib=ref) == want, (chunk, n)
        assert mth_levels(data, chunk) == want, (chunk, n)


def test_commit_of_a_float_tensor_is_its_bytes(ref):
    X = inputs.normal(inputs.rng(902), (300, 77))
    assert oracle.commit(X, 1024, lib=ref) == mth_recursive(X.tobytes(), 1024)
    Y = X.copy()
    Y[123, 45] = np.nextafter(Y[123, 45], np.float32(np.inf))  # one ulp anywhere changes it
    assert oracle.commit(Y, 1024, lib=ref) != oracle.commit(X, 1024, lib=ref)

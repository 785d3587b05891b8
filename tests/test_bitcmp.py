"""The parity checker itself (CPU): a single flipped bit in one output is
reported at its index, signed zeros and NaN payloads are told apart as
documented, and a corrupted input element shows up exactly in the outputs that
depend on it."""
import numpy as np
import pytest

import oracle
from bitcmp import assert_bits_equal, mismatches, ulp_distance
from paper_2502_19405_amd import inputs


def test_one_flipped_bit_is_named_at_its_index():
    g = inputs.rng(1201)
    A, B = inputs.normal(g, (40, 70)), inputs.normal(g, (70, 30))
    C = oracle.matmul(A, B)
    for idx, bit in (((0, 0), 0), ((17, 29), 31), ((39, 5), 22)):
        bad = C.copy()
        bad.view(np.uint32)[idx] ^= np.uint32(1 << bit)
        with pytest.raises(AssertionError) as e:
            assert_bits_equal(bad, C, "flip")
        msg = str(e.value)
        assert f"1 of {C.size} outputs differ" in msg and f"first at {idx}" in msg, msg
        assert list(mismatches(bad, C)) == [np.ravel_multi_index(idx, C.shape)]


def test_signed_zero_and_nan_payloads():
    pz, nz = np.float32(0.0), np.float32(-0.0)
    with pytest.raises(AssertionError):
        assert_bits_equal(np.array([pz]), np.array([nz]), "+0 vs -0")
    q1 = np.array([0x7FC00000], np.uint32).view(np.float32)
    q2 = np.array([0x7FC00001], np.uint32).view(np.float32)
    assert_bits_equal(q1, q2, "NaN class")  # NaN matches NaN by default
    with pytest.raises(AssertionError):
        assert_bits_equal(q1, q2, "NaN payload", nan_equal=False)
    one = np.float32(1.0)
    nxt = np.nextafter(one, np.float32(2.0), dtype=np.float32)
    assert ulp_distance(np.array([one]), np.array([nxt]))[0] == 1
    assert ulp_distance(np.array([nz]), np.array([np.float32(1e-45)]))[0] == 1


def test_corrupted_input_element_shows_in_its_row_only():
    g = inputs.rng(1202)
    A, B = inputs.normal(g, (33, 129)), inputs.normal(g, (129, 65))
    C = oracle.matmul(A, B)
    A2 = A.copy()
    A2[21, 100] = np.nextafter(A2[21, 100], np.float32(np.inf), dtype=np.float32)
    C2 = oracle.matmul(A2, B)
    rows = {int(i) // C.shape[1] for i in mismatches(C2, C)}
    assert rows == {21}

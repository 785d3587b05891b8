"""ISA guard (CPU): the gfx950 assembly of the library's own sources holds none
of the hardware approximations or non-IEEE forms that would make a result
differ from the oracle's fixed binary32 sequence, and the matrix-core path uses
only the single-term fp32 instructions.

- no transcendental approximations (exp, log, rsq, sin, cos): exp, sin/cos and
  1/sqrt are built from basic operations (the paper rebuilds the math functions
  with a controlled order, Section 3.1);
- no unfused multiply-add forms (mad / mac, which round differently from fma)
  and no packed fp32 arithmetic (the build disables it);
- no floating-point atomics (their order of arrival would decide the bits);
- matrix instructions only of the K = 1 kinds, which add one product per step
  (32x32x1 two-block, 16x16x1 four-block, 4x4x1 sixteen-block); the multi-term
  kinds sum several products inside the unit.

Correctly rounded division and square root (v_div_scale / v_div_fmas /
v_div_fixup with v_rcp, and v_sqrt with its correction steps) are IEEE
operations and allowed.
"""
import concurrent.futures
import re

import pytest

from paper_2502_19405_amd import build

SUFFIX = r"(?:_e32|_e64|_dpp|_sdwa)?\b"  # encoding suffixes of a mnemonic
FORBIDDEN = {
    "transcendental approximation": re.compile(
        r"^\s*v_(exp|log|rsq|sin|cos)_(legacy_)?f(16|32|64)" + SUFFIX),
    "unfused multiply-add": re.compile(r"^\s*v_(mad|mac)_(legacy_)?f(16|32)" + SUFFIX),
    "packed fp32 arithmetic": re.compile(r"^\s*v_pk_(fma|mul|add)_f32" + SUFFIX),
    "floating-point atomic": re.compile(
        r"^\s*(global|buffer|flat)_atomic_\w*f(32|64)\b|^\s*ds_(add|sub|min|max)(_rtn)?_f(32|64)\b"),
}
MFMA = re.compile(r"^\s*(v_mfma_\w+)")
SINGLE_TERM = {"v_mfma_f32_32x32x1_2b_f32", "v_mfma_f32_16x16x1_4b_f32", "v_mfma_f32_4x4x1_16b_f32"}


@pytest.fixture(scope="module")
def assembly():
    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        texts = list(ex.map(build.disassemble, build.SOURCES))
    return dict(zip(build.SOURCES, texts))


def instructions(text):
    for line in text.splitlines():
        s = line.strip()
        if s and not s.startswith((";", ".", "//")) and not s.endswith(":"):
            yield line


def scan(text):
    bad = []
    for line in instructions(text):
        for what, pat in FORBIDDEN.items():
            if pat.search(line):
                bad.append(f"{what}: {line.strip()}")
        m = MFMA.match(line)
        if m and m.group(1) not in SINGLE_TERM:
            bad.append(f"multi-term matrix instruction: {line.strip()}")
    return bad


def test_the_guard_flags_each_forbidden_form():
    """The checker itself, on written-out lines (no code is built with them)."""
    flagged = ["v_exp_f32_e32 v1, v2", "v_log_f32 v1, v2", "v_rsq_f32_e32 v3, v4",
               "v_sin_f32_e32 v1, v1", "v_cos_f32 v1, v1", "v_mad_f32 v1, v2, v3, v4",
               "v_mac_f32_e32 v1, v2, v3", "v_mad_legacy_f32 v1, v2, v3, v4",
               "v_pk_fma_f32 v[0:1], v[2:3], v[4:5], v[6:7]", "v_pk_mul_f32 v[0:1], v[2:3], v[4:5]",
               "global_atomic_add_f32 v1, v2, s[0:1]", "ds_add_f32 v1, v2",
               "v_mfma_f32_32x32x2_f32 a[0:15], v1, v2, a[0:15]",
               "v_mfma_f32_16x16x4_f32 a[0:3], v1, v2, a[0:3]"]
    allowed = ["v_fma_f32 v1, v2, v3, v4", "v_fmac_f32_e32 v1, v2, v3", "v_rcp_f32_e32 v1, v2",
               "v_sqrt_f32_e32 v1, v2", "v_div_fixup_f32 v1, v2, v3, v4", "v_ldexp_f32 v1, v2, v3",
               "v_mfma_f32_32x32x1_2b_f32 a[0:31], v1, v2, a[0:31]", "v_exp_legacy_i32 v1, v2",
               "; v_exp_f32 in a comment", "global_atomic_add_u32 v1, v2, s[0:1]"]
    for line in flagged:
        assert scan("\t" + line), line
    for line in allowed:
        assert not scan("\t" + line), line


@pytest.mark.parametrize("src", build.SOURCES)
def test_no_forbidden_instructions(assembly, src):
    bad = scan(assembly[src])
    assert not bad, f"{src}: {len(bad)} forbidden instructions, first: {bad[:3]}"


def test_matrix_core_gemm_uses_the_single_term_instruction(assembly):
    used = {m.group(1) for line in instructions(assembly["gemm_mfma.hip"])
            for m in [MFMA.match(line)] if m}
    assert used == {"v_mfma_f32_32x32x1_2b_f32"}, used

"""Planted mistakes in the oracle must fail its pins (CPU only).

Each case copies the oracle source, plants one plausible mistake by a text
substitution, compiles the copy into a temporary library and runs the pin tests
against it: at least one of the named pins has to fail.  The committed oracle is
never modified.
"""
import os
import tempfile

import pytest

import oracle
import test_oracle as pins
import test_oracle_training as tpins
import test_oracle_llama as lpins
import test_oracle_commit as cpins
import test_oracle_erf as epins

SRC = os.path.join(os.path.dirname(oracle.__file__), "repops_ref.c")

MUTATIONS = {
    # c1: unblocked contraction instead of 64-blocks
    "no_k_blocks": ("const int64_t blk = (k_block > 0) ? k_block : K;", "const int64_t blk = K;",
                    ["w1"]),
    # c1: rounded product then add, in place of the fused update
    "unfused_inner": ("p = fmaf(x, y, p);", "p = p + x * y;", ["w3"]),
    # c1: last term of every block dropped
    "dropped_term": ("for (int64_t k = k0; k < k1; ++k) {", "for (int64_t k = k0; k + 1 < k1; ++k) {",
                     ["int", "bound"]),
    # c1: A read with its transpose's stride
    "transposed_a": ("*inc = 1;\n    return A + i * lda;", "*inc = lda;\n    return A + i;",
                     ["int", "bound"]),
    # c1: block partial not reset between blocks
    "partial_not_reset": ("        float p = 0.0f;\n        for (int64_t k = k0;",
                          "        static __thread float p; if (k0 == 0) p = 0.0f;\n        for (int64_t k = k0;",
                          ["w1", "int", "bound"]),
    # c2: tree partner index off by one
    "tree_index": ("q[l] = q[l] + q[l + s];", "q[l] = q[l] + q[l + s - (s > 1)];", ["w4", "rowint"]),
    # c4: sign of the low part of ln 2 flipped
    "ln2_lo_sign": ("r = fmaf(nf, -EXP_LN2_LO, r);", "r = fmaf(nf, EXP_LN2_LO, r);", ["exp"]),
    # c4: a Taylor coefficient with the wrong exponent (1/12 for 1/24)
    "taylor_coeff": ("0x1.555556p-5f, /* 1/4! */", "0x1.555556p-4f, /* 1/4! */", ["exp"]),
    # c4: a coefficient one ulp off: invisible to accuracy, caught by the
    # constants-against-definitions check
    "taylor_coeff_ulp": ("0x1.555556p-5f, /* 1/4! */", "0x1.555554p-5f, /* 1/4! */", ["const"]),
    # c5: cubic coefficient applied to x^2
    "gelu_power": ("    u = u * x;\n    float z", "    float z", ["gelu"]),
    # c6: max not subtracted (scale-invariant pins still catch it via bits)
    "softmax_no_max": ("const float d = x[j] - m;", "const float d = x[j];", ["softmax_const"]),
    # c7: unbiased variance
    "ln_unbiased": ("const float var = q / nf;", "const float var = q / (nf - 1.0f);", ["ln"]),
    # c7: eps outside the square root
    "ln_eps_outside": ("const float ve = var + c->eps;\n        const float sd = sqrtf(ve);",
                       "const float ve = var + c->eps;\n        const float sd = sqrtf(var) + c->eps;",
                       ["ln"]),
    # softmax backward: sign of the inner product flipped
    "smb_sign": ("const float diff = dy[j] - s;", "const float diff = dy[j] + s;", ["smb", "smb_onehot"]),
    # softmax backward: masked columns get the unmasked formula
    "smb_mask": ("                dx[j] = 0.0f;", "                dx[j] = y[j] * dy[j];", ["smb_causal"]),
    # LayerNorm backward: the t * b projection dropped
    "lnb_no_proj": ("const float w = u - tb;", "const float w = u;", ["lnb"]),
    # LayerNorm backward: gamma not applied to dy
    "lnb_no_gamma": ("t[j] = d * rstd;\n            g[j] = c->gamma ? dy[j] * c->gamma[j] : dy[j];",
                     "t[j] = d * rstd;\n            g[j] = dy[j];", ["lnb"]),
    # LayerNorm parameter gradients: rows summed in one block
    "lnp_unblocked": ("const int64_t blk = c->k_block > 0 ? c->k_block : c->rows;\n    for (int64_t j = j0; j < j1; ++j) {\n        float accg",
                      "const int64_t blk = c->rows;\n    for (int64_t j = j0; j < j1; ++j) {\n        float accg",
                      ["lnp_order"]),
    # LayerNorm parameter gradients: dbeta weighted by t
    "lnp_dbeta_t": ("pb = pb + dy;", "pb = fmaf(dy, t, pb);", ["lnp_int"]),
    # bias gradient: block partial not reset between row blocks
    "colsum_no_reset": ("            float p = 0.0f;\n            for (int64_t i = i0; i < i1; ++i) p = p + c->X",
                        "            static __thread float p; if (i0 == 0) p = 0.0f;\n            for (int64_t i = i0; i < i1; ++i) p = p + c->X",
                        ["colsum"]),
    # GELU backward: (1 - s) factor replaced by s
    "gelu_grad_om": ("const float t2 = t1 * om;", "const float t2 = t1 * s;", ["gelu_grad"]),
    # GELU backward: 3 * 0.044715 coefficient one ulp off
    "gelu_c3_ulp": ("GELU_C3 = 0x1.12ba9ep-3f;", "GELU_C3 = 0x1.12baa0p-3f;", ["tconst"]),
    # Adam: first-moment bias correction missing
    "adam_no_bc1": ("s.step = (float)(dlr / bc1);", "s.step = (float)dlr;", ["adam_sc", "adam"]),
    # Adam: second-moment bias correction multiplied instead of divided
    "adam_bc2_mul": ("const float q = rv / s.sbc2;", "const float q = rv * s.sbc2;", ["adam"]),
    # Adam: coupled weight decay with the wrong sign
    "adam_wd_sign": ("else g = fmaf(s.wd, p, g);", "else g = fmaf(-s.wd, p, g);", ["adam_coupled"]),
    # Adam: binary exponentiation tests the wrong bit
    "adam_pow_bit": ("if (t & 1) result = result * base;", "if (t & 2) result = result * base;",
                     ["adam_sc"]),
    # sin/cos: quadrant 1 mapped like quadrant 3
    "sc_quadrant": ("else if (q == 1) { *sin_out = cv; *cos_out = -sv; }",
                    "else if (q == 1) { *sin_out = -cv; *cos_out = sv; }", ["sc_acc"]),
    # sin/cos: third part of pi/2 dropped
    "sc_no_p3": ("        r = fmaf(n, -SC_P3, r);\n", "", ["sc_acc", "sc_near"]),
    # sin/cos: second part added instead of subtracted
    "sc_p2_sign": ("r = fmaf(n, -SC_P2, r);", "r = fmaf(n, SC_P2, r);", ["sc_acc", "sc_near"]),
    # sin/cos: 1/5! with the exponent of 1/4!
    "sc_coeff": ("SC_S5 = 0x1.111112p-7f;", "SC_S5 = 0x1.111112p-6f;", ["sc_acc"]),
    # sin/cos: a coefficient one ulp off (only the constants check sees it)
    "sc_coeff_ulp": ("SC_C8 = 0x1.a01a02p-16f;", "SC_C8 = 0x1.a01a04p-16f;", ["sc_const"]),
    # rotary embedding: rotation sign flipped
    "rope_sign": ("y[h * c->hd + i] = a - b;", "y[h * c->hd + i] = a + b;", ["rope_acc"]),
    # rotary embedding: position offset ignored
    "rope_offset": ("(c->period > 0 ? r % c->period : r) + c->offset;",
                    "(c->period > 0 ? r % c->period : r);", ["rope_acc"]),
    # rotary embedding: pairs (i, i+1) instead of (i, i + d/2)
    "rope_pairing": ("const float x1 = x[h * c->hd + i], x2 = x[h * c->hd + i + half];",
                     "const float x1 = x[h * c->hd + i], x2 = x[h * c->hd + (i + 1) % c->hd];",
                     ["rope_pairs", "rope_acc"]),
    # RMSNorm: mean of squares over n - 1
    "rms_n1": ("const float ms = q / nf;", "const float ms = q / (nf - 1.0f);", ["rms"]),
    # RMSNorm: eps outside the root
    "rms_eps": ("const float ve = ms + c->eps;\n        const float sd = sqrtf(ve);",
                "const float ve = ms;\n        const float sd = sqrtf(ve) + c->eps;", ["rms"]),
    # RMSNorm backward: projection term dropped
    "rmsb_proj": ("const float w = g[j] - tb;", "const float w = g[j];", ["rmsb"]),
    # RMSNorm dgamma: rows in one block
    "rmsp_unblocked": ("const int64_t blk = c->k_block > 0 ? c->k_block : c->rows;\n    for (int64_t j = j0; j < j1; ++j) {\n        float acc = 0.0f;\n        for (int64_t i0 = 0; i0 < c->rows; i0 += blk) {\n            const int64_t i1 = (i0 + blk < c->rows) ? i0 + blk : c->rows;\n            float pg",
                       "const int64_t blk = c->rows;\n    for (int64_t j = j0; j < j1; ++j) {\n        float acc = 0.0f;\n        for (int64_t i0 = 0; i0 < c->rows; i0 += blk) {\n            const int64_t i1 = (i0 + blk < c->rows) ? i0 + blk : c->rows;\n            float pg",
                       ["rmsp"]),
    # SiLU: exp of +x
    "silu_sign": ("    const float w = -x;\n    const float d = 1.0f + repops_ref_exp1(w);\n    return x / d;",
                  "    const float w = x;\n    const float d = 1.0f + repops_ref_exp1(w);\n    return x / d;",
                  ["silu"]),
    # SiLU derivative: (1 - s) replaced by s
    "silu_grad": ("return fmaf(xs, om, s);", "return fmaf(xs, s, s);", ["silu", "swiglu"]),
    # SwiGLU backward: dup uses g instead of silu(g)
    "swiglu_du": ("const float duv = dyi * repops_ref_silu1(gi);", "const float duv = dyi * gi;",
                  ["swiglu"]),
    # SHA-256: a round constant off by one
    "sha_k": ("0xc67178f2u};", "0xc67178f3u};", ["sha_const", "sha"]),
    # SHA-256: small sigma 0 with the wrong rotation
    "sha_sigma": ("rotr32(W[t - 15], 7)", "rotr32(W[t - 15], 8)", ["sha"]),
    # SHA-256: message length in bytes instead of bits
    "sha_len": ("const uint64_t bits = pos * 8;", "const uint64_t bits = pos;", ["sha"]),
    # commitment: leaves with the internal-node prefix
    "leaf_prefix": ("sha256_prefixed(1, 0x00, data + off, len, out);",
                    "sha256_prefixed(1, 0x01, data + off, len, out);", ["mth"]),
    # commitment: tree split in halves instead of at a power of two
    "mth_split": ("while (k * 2 < count) k *= 2;", "k = count / 2;", ["mth"]),
    # erf: Taylor coefficient with a wrong exponent
    "erf_small_coeff": ("0x1.ce2f22p-4f, -0x1.b82ce4p-6f,", "0x1.ce2f22p-3f, -0x1.b82ce4p-6f,",
                        ["erf"]),
    # erf: one interpolant coefficient one ulp off (only the constants check sees it)
    "erfc_coeff_ulp": ("0x1.71a8d4p-16f", "0x1.71a8d6p-16f", ["erf_const"]),
    # erf: second interval's variable shifted
    "erfc_var": ("const float s = (t - 0.1875f) * 9.5f;", "const float s = (t - 0.1875f) * 9.0f;",
                 ["erf", "gelu_erf"]),
    # exact GELU: x^2 rounded before exp (no split) -- the lower tail loses accuracy
    "erf_no_split": ("    return repops_ref_exp1(a) * repops_ref_exp1(b);",
                     "    return repops_ref_exp1(-(x * x) * c);", ["gelu_erf"]),
    # exact GELU: lower tail through 1 - q
    "phi_branch": ("return x > 0.0f ? 1.0f - q : q;", "return x > 0.0f ? 1.0f - q : 1.0f - (1.0f - q);",
                   ["gelu_erf"]),
    # exact GELU derivative: pdf term without the 1/sqrt(2 pi)
    "gelu_erf_grad": ("const float phi = e * ERF_INV_SQRT_2PI;", "const float phi = e;",
                      ["gelu_erf_grad"]),
}

CHECKS = {
    "const": lambda lib: pins.check_constants(open(lib._name[:-len("mutant.so")] + "repops_ref.c").read()),
    "w1": lambda lib: pins.test_witness_w1_blocked_vs_sequential(lib),
    "w3": lambda lib: pins.test_witness_w3_fused_vs_unfused(lib),
    "w4": lambda lib: pins.test_witness_w4_strided_tree(lib),
    "int": lambda lib: pins.test_matmul_integer_closed_form(lib, (19, 23, 65), 0, 0, 64, 0),
    "bound": lambda lib: pins.test_matmul_error_bound(lib, 200, 64),
    "rowint": lambda lib: pins.test_rowsum_integers_exact(lib, 100, 64, 0),
    "exp": lambda lib: pins.test_exp_accuracy_under_one_ulp(lib),
    "gelu": lambda lib: pins.test_gelu_accuracy_bound(lib),
    "softmax_const": lambda lib: pins.test_softmax_constant_row_is_reciprocal(lib),
    "ln": lambda lib: pins.test_layernorm_bound(lib, 3e-3),
    "smb": lambda lib: tpins.test_softmax_backward_bound(lib, 64, 0),
    "smb_onehot": lambda lib: tpins.test_softmax_backward_one_hot_closed_form(lib),
    "smb_causal": lambda lib: tpins.test_softmax_backward_causal_masked_zero(lib),
    "lnb": lambda lib: tpins.test_layernorm_backward_bound(lib),
    "lnp_order": lambda lib: tpins.test_layernorm_param_grads_order_witness(lib),
    "lnp_int": lambda lib: tpins.test_layernorm_param_grads_integer_exact(lib),
    "gelu_grad": lambda lib: tpins.test_gelu_grad_bound(lib),
    "colsum": lambda lib: tpins.test_colsum_witness_and_integers(lib),
    "tconst": lambda lib: tpins.check_training_constants(
        open(lib._name[:-len("mutant.so")] + "repops_ref.c").read()),
    "adam_sc": lambda lib: tpins.test_adam_scalars(lib),
    "adam": lambda lib: tpins.test_adam_against_float64(lib, 0.0, False),
    "adam_coupled": lambda lib: tpins.test_adam_against_float64(lib, 0.01, False),
    "sc_acc": lambda lib: lpins.test_sincos_accuracy(lib, 4096.0),
    "sc_near": lambda lib: lpins.test_sincos_near_multiples_of_half_pi(lib),
    "sc_const": lambda lib: lpins.check_sincos_constants(
        open(lib._name[:-len("mutant.so")] + "repops_ref.c").read()),
    "rope_acc": lambda lib: lpins.test_rope_rotation_accuracy_and_inverse(lib),
    "rope_pairs": lambda lib: lpins.test_rope_pairs_rotate_half(lib),
    "rms": lambda lib: lpins.test_rmsnorm_bound(lib, 64, 0),
    "rmsb": lambda lib: lpins.test_rmsnorm_backward_bound(lib),
    "rmsp": lambda lib: lpins.test_rmsnorm_dgamma_order_witness_and_integers(lib),
    "silu": lambda lib: lpins.test_silu_and_grad_bounds(lib),
    "swiglu": lambda lib: lpins.test_swiglu_forward_and_backward(lib),
    "sha": lambda lib: cpins.test_sha256_every_length_against_hashlib(lib),
    "sha_const": lambda lib: cpins.check_sha_constants(
        open(lib._name[:-len("mutant.so")] + "repops_ref.c").read()),
    "mth": lambda lib: cpins.test_commit_against_rfc6962(lib, 64),
    "erf": lambda lib: epins.test_erf_accuracy_and_symmetry(lib),
    "erf_const": lambda lib: epins.check_erf_constants(
        open(lib._name[:-len("mutant.so")] + "repops_ref.c").read()),
    "gelu_erf": lambda lib: epins.test_gelu_erf_accuracy(lib),
    "gelu_erf_grad": lambda lib: epins.test_gelu_erf_grad(lib),
}


def _build_mutant(tmp, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    path = os.path.join(tmp, "repops_ref.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    hdr = os.path.join(os.path.dirname(SRC), "repops_ref.h")
    with open(os.path.join(tmp, "repops_ref.h"), "w") as f:
        f.write(open(hdr).read())
    import subprocess
    out = os.path.join(tmp, "mutant.so")
    subprocess.run(["gcc", *oracle.CFLAGS, "-o", out, path, "-lm", "-lpthread"], check=True)
    return oracle.load(out)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name):
    old, new, checks = MUTATIONS[name]
    with tempfile.TemporaryDirectory() as tmp:
        lib = _build_mutant(tmp, old, new)
        caught = []
        for c in checks:
            try:
                CHECKS[c](lib)
            except AssertionError:
                caught.append(c)
        assert caught, f"mutation {name} passed every pin in {checks}"


def test_unmutated_copy_passes_the_same_checks():
    with tempfile.TemporaryDirectory() as tmp:
        lib = _build_mutant(tmp, "#include <fenv.h>", "#include <fenv.h>")
        for fn in CHECKS.values():
            fn(lib)

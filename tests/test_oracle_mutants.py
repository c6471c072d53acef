"""The oracle's pins must catch plausible mistakes.

Each case copies the oracle's C source, plants one mistake by a text
substitution, builds the altered copy into a temporary library and runs the
pins of test_oracle_pins.py against it: at least one pin must fail.  Only the
CPU is involved; the real oracle library is untouched.
"""
import os
import shutil
import tempfile

import pytest

import test_oracle_pins as pins
from oracle import build as obuild
from oracle import oracle as O

MUTANTS = [
    ("scale divisor Q+1",
     "absmax / (double)Q", "absmax / (double)(Q + 1)"),
    ("code ties away from zero",
     "rint((double)w[j] / s)", "round((double)w[j] / s)"),
    ("no clamp of codes",
     "if (r > Q)\n                r = Q;", ""),
    ("max instead of absmax",
     "if (fabs(v) > absmax)", "if (v > absmax)"),
    ("NaN/Inf not rejected",
     "if (!isfinite(v))\n            return ORC_ERR_RANGE;", ""),
    ("fp16 encode rounds half up",
     "rint(ldexp(a, 10 - E))", "floor(ldexp(a, 10 - E) + 0.5)"),
    ("fp16 encode subnormal threshold",
     "if (a < 0x1p-14) {", "if (a < 0x1p-15) {"),
    ("fp16 decode exponent bias",
     "ldexp((double)(man + 1024), ex - 25)", "ldexp((double)(man + 1024), ex - 24)"),
    ("q4 nibbles stored swapped",
     "    if (k & 1)\n        *p", "    if (!(k & 1))\n        *p"),
    ("q4 code read unsigned",
     "return nib >= 8 ? nib - 16 : nib;", "return nib;"),
    ("forward drops the block scale",
     "y += oracle_f16_to_f64(scales[n * nb + b]) * partial;", "y += partial;"),
    ("forward uses the first block's scale for all",
     "y += oracle_f16_to_f64(scales[n * nb + b]) * partial;",
     "y += oracle_f16_to_f64(scales[n * nb]) * partial;"),
    ("forward shifted activation index",
     "partial += x_at(X, xdt, K, m, k)", "partial += x_at(X, xdt, K, m, (k + 1) % K)"),
    ("forward reads the next block's codes",
     "code_at(fmt, codes, K, n, k);\n        }", "code_at(fmt, codes, K, n, (k + ORC_BLOCK) % K);\n        }"),
    ("bf16 decode shift",
     "(uint32_t)b << 16", "(uint32_t)b << 15"),
    ("fp16-weight forward transposed weight index",
     "oracle_f16_to_f64(W[n * K + k])", "oracle_f16_to_f64(W[k * N + n])"),
    ("fp16-weight forward shifted activation index",
     "y += x_at(X, xdt, K, m, k) * oracle_f16_to_f64(W",
     "y += x_at(X, xdt, K, m, (k + 1) % K) * oracle_f16_to_f64(W"),
    ("fp16-weight forward ignores the row list",
     "const int64_t m = rows ? rows[i] : i;", "const int64_t m = i;"),
    ("GELU without the 1/sqrt(2)",
     "erf(v / sqrt(2.0))", "erf(v)"),
    ("epilogue bias indexed by row",
     "v += (double)bias[n];", "v += (double)bias[i % N];"),
    ("epilogue residual before the activation",
     "            if (act == ORC_ACT_GELU)\n                v = v * 0.5 * (1.0 + erf(v / sqrt(2.0)));\n            if (residual)\n                v += (double)residual[src * N + n];",
     "            if (residual)\n                v += (double)residual[src * N + n];\n            if (act == ORC_ACT_GELU)\n                v = v * 0.5 * (1.0 + erf(v / sqrt(2.0)));"),
    ("epilogue residual ignores the row list",
     "v += (double)residual[src * N + n];", "v += (double)residual[i * N + n];"),
    ("attention ignores the scale",
     "const double p = exp(scale * dot - smax);", "const double p = exp(dot - smax);"),
    ("attention weights values by the key rows",
     "out[c] += p * oracle_bf16_to_f64(V[(b * T + j) * ldv + h * dh + c]);",
     "out[c] += p * oracle_bf16_to_f64(K[(b * T + j) * ldk + h * dh + c]);"),
    ("attention keys from the first sequence",
     "oracle_bf16_to_f64(K[(b * T + j) * ldk + h * dh + c]);\n                const double p",
     "oracle_bf16_to_f64(K[j * ldk + h * dh + c]);\n                const double p"),
    ("attention heads share head 0's queries",
     "                    dot += oracle_bf16_to_f64(Q[r * ldq + h * dh + c]) *\n                           oracle_bf16_to_f64(K[(b * T + j) * ldk + h * dh + c]);\n                const double p",
     "                    dot += oracle_bf16_to_f64(Q[r * ldq + c]) *\n                           oracle_bf16_to_f64(K[(b * T + j) * ldk + h * dh + c]);\n                const double p"),
    ("attention not normalized",
     "                out[c] /= denom;", "                out[c] /= (double)T;"),
    ("steering ignores the residual norm",
     "const double c = alpha * hnorm;", "const double c = alpha;"),
    ("steering applied at zero strength",
     "    if (alpha == 0.0)\n        return ORC_OK;\n    const double c", "    const double c"),
    ("steering indexes the direction by row",
     "Y[i * N + n] += c * (double)dir[n];", "Y[i * N + n] += c * (double)dir[(i + n) % N];"),
    ("activation scale divisor 128",
     "absmax / 127.0", "absmax / 128.0"),
    ("activation codes round half away from zero",
     "rint(x_at(X, xdt, K, m, k) / sv)", "round(x_at(X, xdt, K, m, k) / sv)"),
    ("activation absmax ignores negative values",
     "            else if (absmax < fabs(v))\n                absmax = fabs(v);",
     "            else if (absmax < v)\n                absmax = v;"),
    ("W8A8 forward drops the activation scale",
     "Y[i * N + n] = oracle_f16_to_f64(sx[row]) * y;", "Y[i * N + n] = y;"),
    ("W8A8 forward uses the first row's scale",
     "Y[i * N + n] = oracle_f16_to_f64(sx[row]) * y;", "Y[i * N + n] = oracle_f16_to_f64(sx[0]) * y;"),
    ("W8A8 forward reads the next block's weight codes",
     "(int64_t)code_at(ORC_FMT_INT8, codes, K, n, k);",
     "(int64_t)code_at(ORC_FMT_INT8, codes, K, n, (k + 32) % K);"),
]


def pin_cases():
    F = [O.FMT_INT8, O.FMT_Q4]
    cases = []
    cases += [(pins.test_range_errors, (f,)) for f in F]
    cases += [(pins.test_shape_errors, ())]
    cases += [(pins.test_q4_packing_layout, ())]
    cases += [(pins.test_half_integer_ties_go_to_even, ())]
    cases += [(pins.test_power_of_two_weights_exact, (f,)) for f in F]
    cases += [(pins.test_unit_scale_integer_matmul, (f,)) for f in F]
    cases += [(pins.test_invariants_roundtrip_maxcode_idempotent, (f,)) for f in F]
    cases += [(pins.test_forward_matches_dequantized_matmul, (f, x)) for f in F for x in (0, 1)]
    cases += [(pins.test_forward_bruteforce_tiny, (f, 32)) for f in F]
    cases += [(pins.test_bf16_decode, ())]
    cases += [(pins.test_scales_and_codes_bruteforce, (f,)) for f in F]
    cases += [(pins.test_f16_encode_special_values, ())]
    cases += [(pins.test_f16_decode_all_patterns, ())]
    cases += [(pins.test_f16_encode_exact_values_roundtrip, ())]
    cases += [(pins.test_f16_encode_midpoints_and_neighbours, ())]
    cases += [(pins.test_forward_f16_integer_bruteforce, (x,)) for x in (0, 1)]
    cases += [(pins.test_forward_f16_equals_quantized_at_power_of_two_scales, (f,)) for f in F]
    cases += [(pins.test_forward_f16_subnormal_and_signed_zero_weights, ())]
    cases += [(pins.test_epilogue_gelu_normal_cdf_values, ())]
    cases += [(pins.test_epilogue_bias_residual_exact_and_order, ())]
    cases += [(pins.test_attention_zero_queries_average_values, ())]
    cases += [(pins.test_attention_single_key_returns_its_value, ())]
    cases += [(pins.test_attention_two_keys_sigmoid, ())]
    cases += [(pins.test_attention_dominant_key, ())]
    cases += [(pins.test_attention_key_permutation_and_heads, ())]
    cases += [(pins.test_steer_zero_strength_is_identity, ())]
    cases += [(pins.test_steer_rank_one_shift, ())]
    cases += [(pins.test_act_quant_bruteforce, (x,)) for x in (0, 1)]
    cases += [(pins.test_act_quant_equals_weight_quantizer_one_block, ())]
    cases += [(pins.test_act_quant_invariants, ())]
    cases += [(pins.test_act_quant_range_errors, ())]
    cases += [(pins.test_forward_w8a8_integer_exact, ())]
    cases += [(pins.test_forward_w8a8_matches_dequantized_matmul, ())]
    cases += [(pins.test_forward_w8a8_exact_rationals_tiny, ())]
    return cases


@pytest.fixture(scope="module")
def tmpdir_mut():
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmpdir_mut, name, old, new):
    src = open(obuild.SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/found: {old!r}"
    tag = "".join(ch if ch.isalnum() else "_" for ch in name)
    csrc = os.path.join(tmpdir_mut, f"{tag}.c")
    lib = os.path.join(tmpdir_mut, f"lib{tag}.so")
    with open(csrc, "w") as f:
        f.write(src.replace(old, new))
    obuild.build(src=csrc, out=lib, extra_flags=("-w",))
    mut = O.Oracle(lib)
    for fn, args in pin_cases():
        try:
            fn(mut, *args)
        except (AssertionError, O.OracleError, ValueError, IndexError, OverflowError):
            return  # caught
    pytest.fail(f"no pin caught the planted mistake: {name}")

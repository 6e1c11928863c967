"""Planted mistakes in the oracle (on the CPU): each broken copy of
dfssm_ref.c must fail at least one pin.  This is what shows the pins can
catch a dropped term, a wrong sign, a wrong index or a transposed operand."""
import os

import pytest

import oracle
from oracle import Oracle
from oracle_pins import ALL_PINS

# (name, [(original text, replacement), ...]) -- every original must occur
# exactly once in dfssm_ref.c
MUTANTS = [
    ("bit_order_msb_first", [("(word >> (k % 32))", "(word >> (31 - k % 32))")]),
    ("sign_polarity", [("? +1 : -1", "? -1 : +1")]),
    ("drop_lora_term", [("if (r > 0) d = d + (double)beta[n] * (double)sb;", "(void)sb;"),
                        ("w = u + v;", "w = u; (void)v;")]),
    ("A_transposed", [("(int64_t)A[j * K + k]", "(int64_t)A[(k % r) * K + (k / r) % K]")]),
    ("B_transposed", [("(int64_t)B[n * r + j]", "(int64_t)B[j * N + n]")]),
    ("lora_down_row0", [("(int64_t)A[j * K + k] * (int64_t)q[m * K + k]", "(int64_t)A[j * K + k] * (int64_t)q[k]")]),
    ("round_half_away", [("float rq = rintf(t);", "float rq = roundf(t);")]),
    ("scale_over_128", [("s[m] = a / 127.0f;", "s[m] = a / 128.0f;")]),
    ("inv_from_s", [("float inv = 127.0f / a;", "float inv = 1.0f / (a / 127.0f);")]),
    ("acc_b_int32", [("int64_t sb = 0;", "int32_t sb = 0;")]),
    ("acc_a_int16", [("a_buf[m * r + j] = (int32_t)sum;", "a_buf[m * r + j] = (int16_t)sum;")]),
    ("f16_bias", [("(1024 + f), e - 25)", "(1024 + f), e - 24)")]),
    ("f16_subnormal", [("ldexpf((float)f, -24)", "ldexpf((float)f, -25)")]),
    ("y_missing_s", [("y32[m * N + n] = s[m] * w;", "y32[m * N + n] = w;"),
                     ("y64[m * N + n] = (double)s[m] * d;", "y64[m * N + n] = d;")]),
    ("alpha_row0", [("float u = alpha[n] * fs;", "float u = alpha[0] * fs;"),
                    ("double d = (double)alpha[n] * (double)ss;", "double d = (double)alpha[0] * (double)ss;")]),
    ("fma_in_epilogue", [("w = u + v;", "w = fmaf(beta[n], fb, u); (void)v;")]),
    ("absmax_over_stride", [("for (int64_t k = 0; k < K; ++k) {\n      float v = load_x(x, x_dtype, m * ldx + k);\n      if (!isfinite(v))",
                             "for (int64_t k = 0; k < ldx; ++k) {\n      float v = load_x(x, x_dtype, m * ldx + k);\n      if (!isfinite(v))")]),
    ("zero_row_unit_scale", [("if (a < FLT_MIN) {\n      s[m] = 0.0f;", "if (a < FLT_MIN) {\n      s[m] = 1.0f;")]),
    ("chain_keeps_scale", [("for (int64_t m = 0; m < M; ++m) sbuf[m] = 1.0f / 127.0f;", "(void)0;")]),
    ("chain_wrong_prefix_stride", [("N[l - 1], qbuf, sbuf);", "K[l], qbuf, sbuf);")]),
    ("lm_head_scale_row0", [("float t = scale[v] * fa;", "float t = scale[0] * fa;")]),
    ("lm_head_missing_s", [("logits[m * V + v] = s[m] * t;", "logits[m * V + v] = t;")]),
    ("lm_head_scale_order", [("float t = scale[v] * fa;\n        logits[m * V + v] = s[m] * t;",
                              "float t = s[m] * fa;\n        logits[m * V + v] = scale[v] * t;")]),
    ("lm_head_E_transposed", [("(int64_t)E[v * d + k] * (int64_t)q[m * d + k]",
                               "(int64_t)E[(k % V) * d + (v % d)] * (int64_t)q[m * d + k]")]),
    ("lm_head_acc_int16", [("if (acc) acc[m * V + v] = (int32_t)sum;", "if (acc) acc[m * V + v] = (int16_t)sum;")]),
    ("embed_row_of_m", [("x[m * d + k] = scale[v] * (float)E[v * d + k];", "x[m * d + k] = scale[v] * (float)E[m * d + k];")]),
    # the Mamba-2 step around the linears (Table 12's three fixes first)
    ("ssm_missing_dt", [("const float dtx = dt * x;", "const float dtx = x;")]),
    ("gate_after_norm", [("g[k] = y[m * d + k] * silu_f(z[m * ldz + k]);", "g[k] = y[m * d + k];"),
                         ("on[m * d + k] = (g[k] * r) * w[k];",
                          "on[m * d + k] = ((g[k] * r) * w[k]) * silu_f(z[m * ldz + k]);")]),
    ("ssm_state_head0", [("float* hs = ssm_state + ((m * H + h) * P + p) * N;",
                          "float* hs = ssm_state + ((m * H + 0) * P + p) * N;")]),
    ("conv_taps_reversed", [("float v = wc[0] * st[0];", "float v = wc[3] * st[0];"),
                            ("v = v + wc[3] * st[3];", "v = v + wc[0] * st[3];")]),
    ("conv_no_shift", [("      st[0] = st[1];\n      st[1] = st[2];\n      st[2] = st[3];\n", "")]),
    ("conv_no_bias", [("v = v + conv_b[c];", "(void)0;")]),
    ("A_positive", [("(float)(-exp((double)A_log[h]))", "(float)(exp((double)A_log[h]))")]),
    ("no_softplus", [("const float dt = softplus_f(row[d_inner + conv_dim + h] + dt_bias[h]);",
                      "const float dt = row[d_inner + conv_dim + h] + dt_bias[h];")]),
    ("missing_D", [(" + (double)D[h] * (double)x)", ")")]),
    ("B_C_swapped", [("const float* Bv = c_out + d_inner;", "const float* Bv = c_out + d_inner + N;"),
                     ("const float* Cv = c_out + d_inner + N;", "const float* Cv = c_out + d_inner;")]),
    ("norm_no_eps", [("sqrt(ss / (double)d + (double)eps)", "sqrt(ss / (double)d)")]),
    ("norm_sum_not_mean", [("sqrt(ss / (double)d + (double)eps)", "sqrt(ss + (double)eps)")]),
    ("int4_high_nibble_first", [("const int nib = (i % 2 == 0) ? (byte & 0x0f) : (byte >> 4);",
                                 "const int nib = (i % 2 == 0) ? (byte >> 4) : (byte & 0x0f);")]),
    ("int4_unsigned", [("out[i] = (int8_t)(nib >= 8 ? nib - 16 : nib);", "out[i] = (int8_t)nib;")]),
    ("int4_minus8_as_8", [("out[i] = (int8_t)(nib >= 8 ? nib - 16 : nib);", "out[i] = (int8_t)(nib > 8 ? nib - 16 : nib);")]),
    ("residual_dropped", [("res[k] = delta ? u[m * d + k] + delta[m * d + k] : u[m * d + k];", "res[k] = u[m * d + k];")]),
]


@pytest.mark.parametrize("name,edits", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, edits):
    src = open(oracle.SRC).read()
    for old, new in edits:
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
    c = tmp_path / "dfssm_ref.c"
    c.write_text(src)
    so = str(tmp_path / f"libref_{name}.so")
    oracle.build(src=str(c), out=so, extra=["-Wno-unused-variable", "-Wno-unused-but-set-variable", "-Wno-unused-function", "-Wno-unused-parameter"])
    o = Oracle(so)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(o)
        except (AssertionError, oracle.OracleError):
            failed.append(pin.__name__)
    assert failed, f"planted mistake {name} passed every pin"

"""The oracle's pins must catch plausible mistakes.

Each case plants one slip (a dropped term, a wrong sign, a wrong index, a
transposed operand, a garbled formula read literally) in a copy of the oracle's
C source, builds that copy on the CPU, and runs the pin suite against it: the
suite must fail.  Nothing here touches the GPU or the HIP library.
"""
import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "fqvit_oracle.c")

# (name, original text, planted mistake)
MUTANTS = [
    ("ptf_shift_direction", "(XQ - zp) * ((int64_t)1 << a)", "(XQ - zp) * ((int64_t)1 << (K - a))"),
    ("ptf_zero_point_dropped", "Xh[i] = (XQ - zp) *", "Xh[i] = (XQ) *"),
    ("variance_sign", "(int64_t)C * M2 - M1 * M1", "(int64_t)C * M2 + M1 * M1"),
    ("variance_sqrt_dropped", "const double D = sqrt((double)Vr);", "const double D = (double)Vr;"),
    ("B_sign", "B = bs - gs * m;", "B = bs + gs * m;"),
    ("r_transposed", "const double r = (double)C / D;", "const double r = D / (double)C;"),
    ("mean_uses_M2", "const double m = (double)M1 / D;", "const double m = (double)M2 / D;"),
    ("N1_off_by_one", "(int64_t)bits - 1 - (int64_t)ilogb", "(int64_t)bits - (int64_t)ilogb"),
    ("outer_round_dropped", "floor_div(y + ((int64_t)1 << (N1 - 1)),", "floor_div(y,"),
    ("zp_out_dropped", "clip_i64(w + zp_o, 0, levels)", "clip_i64(w, 0, levels)"),
    ("ln_sign_dropped", "const int64_t y = sgn * N2 * Xh[i] + Bq;", "const int64_t y = N2 * Xh[i] + Bq;"),
    ("q_ln2_ceil", "(int64_t)floor(-LN2 / s)", "(int64_t)ceil(-LN2 / s)"),
    ("q_c_missing_s", "IEXP_C / ((IEXP_A * s) * s)", "IEXP_C / (IEXP_A * s)"),
    ("q_L_as_printed", "const int64_t w = k->q_b - r;", "const int64_t w = k->q_b - u;"),
    ("q_c_dropped", "const int64_t poly = w * w + k->q_c;", "const int64_t poly = w * w;"),
    ("exp_shift_direction", "return poly << (k->n - z);", "return poly << z;"),
    ("clamp_dropped", "const int64_t u = -q < u_max ? -q : u_max;",
     "const int64_t u = -q < 2 * u_max ? -q : 2 * u_max;"),
    ("max_not_subtracted", "e[j] = oracle_iexp(v[j] - vmax, k, NULL, NULL);",
     "e[j] = oracle_iexp(v[j] - v[0], k, NULL, NULL);"),
    ("q_rev_floor", "(2 * S + ej) / (2 * ej)", "(2 * S) / (2 * ej)"),
    ("ilog2_rounds_at_1_25", "(unsigned __int128)2 * r >= ((unsigned __int128)3 << M)",
     "(unsigned __int128)4 * r >= ((unsigned __int128)5 << M)"),
    ("ilog2_round_bit_dropped", "return M + round_up;", "return M;"),
    ("code_clip_dropped", "code[j] = lg < top ? lg : top;", "code[j] = lg & top;"),
    ("nibble_order", "(uint8_t)(lo | (hi << 4))", "(uint8_t)(hi | (lo << 4))"),
    ("bias_wrong_head", "bias + ((g % Hb) * Lq + i)", "bias + ((g / Hb % Hb) * Lq + i)"),
    ("av_zp_dropped", "(int64_t)v[(g * Lk + j) * (int64_t)d + c] - zp_v;", "(int64_t)v[(g * Lk + j) * (int64_t)d + c];"),
    ("av_shift_is_code", "((int64_t)1 << (shift < 0 ? 0 : shift))", "((int64_t)1 << attn_q)"),
    ("av_v_transposed", "v[(g * Lk + j) * (int64_t)d + c]", "v[(g * d + c) * (int64_t)Lk + j]"),
    ("ptf_scale_times_2K", "(mx - mn) / levels / two_K", "(mx - mn) / levels * two_K"),
    ("ptf_quant_neg_alpha", "x / (ldexp(1.0, alpha) * s)", "x / (ldexp(1.0, -alpha) * s)"),
    ("minmax_zp_sign", "round_nearest(-l / *s)", "round_nearest(l / *s)"),
    ("alpha_last_row_dropped", "for (int64_t t = 0; t < T; ++t) {\n                const double xv",
     "for (int64_t t = 0; t < T - 1; ++t) {\n                const double xv"),
    ("alpha_deq_zp_dropped", "ptf_q(xv, s, zp, a, levels) - (double)zp, step)",
     "ptf_q(xv, s, zp, a, levels), step)"),
    ("alpha_argmax", "if (xacc_cmp(&acc[a], &acc[best]) < 0) best = a;",
     "if (xacc_cmp(&acc[a], &acc[best]) > 0) best = a;"),
    ("alpha_cross_terms_halved", "const double f = (i == j) ? 1.0 : 2.0;",
     "const double f = (i == j) ? 1.0 : 1.0;"),
    ("alpha_residual_low_part_dropped", "const double t[3] = {u, ul, -pl};",
     "const double t[3] = {u, 0.0, -pl};"),
    ("alpha_product_rounded", "xacc_add(acc, f * h);\n            xacc_add(acc, f * l);",
     "xacc_add(acc, f * h + f * l);"),
    ("requant_precision_16", "int64_t N1 = 31 - (int64_t)e;", "int64_t N1 = 16 - (int64_t)e;"),
    ("requant_round_down", "(prod + ((__int128)1 << (N1 - 1))) >> N1", "prod >> N1"),
    ("requant_zp_dropped", "const __int128 yu = w + zp;", "const __int128 yu = w + half;"),
    ("requant_inverse_scale", "(double)s_in / (double)s_out", "(double)s_out / (double)s_in"),
    ("qk_zero_point_sign", "((int64_t)qi[c] - zp_q)", "((int64_t)qi[c] + zp_q)"),
    ("qk_zp_k_dropped", "((int64_t)kj[c] - zp_k)", "((int64_t)kj[c])"),
    ("qk_k_transposed", "k + (g * Lk + j) * (int64_t)dk", "k + (g * Lk + j)"),
    ("wide_codes_truncated", "out[j] = (uint8_t)code[j];", "out[j] = (uint8_t)(code[j] & 15);"),
]


def _run_mutant(name, old, new, tmp):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"{name}: pattern not found in the oracle source"
    mutated = src.replace(old, new)
    csrc = os.path.join(tmp, f"{name}.c")
    so = os.path.join(tmp, f"{name}.so")
    with open(csrc, "w") as f:
        f.write(mutated)
    sys.path.insert(0, ROOT)
    import oracle
    oracle.build(src=csrc, out=so)
    env = dict(os.environ, FQVIT_ORACLE_LIB=so, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(HERE, "test_oracle_pins.py"),
                        "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode


def test_every_planted_mistake_is_caught():
    with tempfile.TemporaryDirectory() as tmp:
        workers = min(8, os.cpu_count() or 2)
        with cf.ThreadPoolExecutor(workers) as ex:
            results = list(ex.map(lambda m: _run_mutant(*m, tmp), MUTANTS))
    survivors = [n for n, rc in results if rc == 0]
    assert not survivors, f"mutants not caught by the pins: {survivors}"

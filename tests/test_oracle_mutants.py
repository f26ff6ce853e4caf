"""Planted mistakes: each test builds a copy of the oracle with one plausible bug and checks
that the CPU pin suite catches it.  The mistakes are planted in the oracle only, on the CPU."""
import os
import subprocess
import sys
from pathlib import Path

import pytest

import oracle

ROOT = Path(__file__).resolve().parents[1]

# (name, original text, planted text): every original must occur exactly once.
# Rounding s_base to the nearest FP8 value instead of down moves the window up by one code
# exactly when max|y| / 6 lies above an FP8 midpoint.  For a normal base code the extra top
# code loses to its half inside the window (Lemma 1, which needs s / 2 on the FP8 grid), but
# for the odd subnormal codes 1..7 it does not, and tests/test_oracle_subnormal.py holds blocks
# whose code changes; the two "nearest" mutants below plant the mistake in the selection and in
# the window-variant path.
MUTANTS = [
    ("fp4_tie_rule", "if (a > mid || (a == mid && ((k + 1) % 2) == 0))",
     "if (a > mid || (a == mid && ((k + 1) % 2) == 1))"),
    ("fp8_tie_rule", "if (v_num > mid || (v_num == mid && ((c + 1) % 2) == 0)) c++;",
     "if (v_num > mid || (v_num == mid && ((c + 1) % 2) == 1)) c++;"),
    ("window_upper_6", "int nvfp4_ref_window_upper(void) { return 7; }",
     "int nvfp4_ref_window_upper(void) { return 6; }"),
    ("mse_lower_2", "int mse = (n == 16) ? 3 :", "int mse = (n == 16) ? 2 :"),
    ("wmse_lower_7", "return mse > 8 ? mse : 8;", "return mse > 7 ? mse : 7;"),
    ("weight_dropped", "if (w) t = (double)w[i] * t;", "if (0) t = (double)w[i] * t;"),
    ("abs_error_not_squared", "double t = e * e;", "double t = fabs(e);"),
    ("eemm_bias_off_by_one", "int bias = (1 << (e - 1)) - 1;", "int bias = (1 << (e - 1));"),
    ("fp8_floor_strictness", "while (c > 0 && v_den * nvfp4_ref_e4m3(c) > v_num) c--;",
     "while (c > 0 && v_den * nvfp4_ref_e4m3(c) >= v_num) c--;"),
    ("argmin_tie_largest_code", "if (J < jb) { best = c; jb = J; }",
     "if (J <= jb) { best = c; jb = J; }"),
    ("sign_dropped", "int nib = (signbit(y[i]) ? 8 : 0) | k;", "int nib = k;"),
    ("dequant_nibble_order", "int nib = (e & 1) ? (q[e >> 1] >> 4) : (q[e >> 1] & 15);",
     "int nib = (e & 1) ? (q[e >> 1] & 15) : (q[e >> 1] >> 4);"),
    ("global_scale_uses_4", "float denom = 6.0f * fp8_range;", "float denom = 4.0f * fp8_range;"),
    ("four_over_six_tie_to_4", "return (j4 < j6) ? c4 : c6;", "return (j4 <= j6) ? c4 : c6;"),
    ("four_over_six_uses_3", "int c4 = nvfp4_ref_nearest_fp8(ymax, 4.0);",
     "int c4 = nvfp4_ref_nearest_fp8(ymax, 3.0);"),
    ("normalize_by_reciprocal", "y[i] = v / S;", "y[i] = v * (1.0f / S);"),
    ("s0_rounds_to_nearest_in_sweep",
     "double ymax = block_ymax(y, n);\n    int c0 = nvfp4_ref_floor_fp8(ymax, 6.0);",
     "double ymax = block_ymax(y, n);\n    int c0 = nvfp4_ref_nearest_fp8(ymax, 6.0);"),
    ("s_base_nearest_in_selection",
     "int U = nvfp4_ref_window_upper();\n    int c0 = nvfp4_ref_floor_fp8(ymax, 6.0);",
     "int U = nvfp4_ref_window_upper();\n    int c0 = nvfp4_ref_nearest_fp8(ymax, 6.0);"),
    ("window_base_nearest",
     "int c0 = nvfp4_ref_floor_fp8(block_ymax(y, block), 6.0);",
     "int c0 = nvfp4_ref_nearest_fp8(block_ymax(y, block), 6.0);"),
    ("window_not_clamped_to_1", "int lo = c0 - L < 1 ? 1 : c0 - L;\n    int hi = c0 + U > E4M3_MAX_CODE ? E4M3_MAX_CODE : c0 + U;\n    const float* wm",
     "int lo = c0 - L < 0 ? 0 : c0 - L;\n    int hi = c0 + U > E4M3_MAX_CODE ? E4M3_MAX_CODE : c0 + U;\n    const float* wm"),
    ("zero_tensor_scale", "        *S = 1.0f;\n        return REF_OK;", "        *S = 0.5f;\n        return REF_OK;"),
    ("tight_lower_strict", "5.0 * nvfp4_ref_e4m3(c_inf - 1) >= 4.0 * s0",
     "5.0 * nvfp4_ref_e4m3(c_inf - 1) > 4.0 * s0"),
    ("tight_upper_from_s0", "*upper = nvfp4_ref_floor_fp8(12.0 * s1, 7.0) - c0;",
     "*upper = nvfp4_ref_floor_fp8(12.0 * s0, 7.0) - c0;"),
    ("window_clamp_to_0", "*lo = l < 1 ? 1 : l > E4M3_MAX_CODE", "*lo = l < 0 ? 0 : l > E4M3_MAX_CODE"),
    ("window_offsets_mirrored", "int l = c0 + lo_off, h = c0 + hi_off;",
     "int l = c0 - hi_off, h = c0 - lo_off;"),
    ("swizzle_row_split", "(mm % 32) * 16 + (mm / 32) * 4", "(mm / 4) * 16 + (mm % 4) * 4"),
    ("norm_group_div_dropped", "int64_t g = ((r / group_rows) % groups) / group_div;",
     "int64_t g = ((r / group_rows) % groups) % (groups / group_div);"),
    ("online_group_index", "importance + ((r / imp_group_rows) % imp_groups) * cols",
     "importance + (r % imp_groups) * cols"),
    ("optimum_piece_at_low_end", "double s_ref = (seg == 0) ? 0.5 * hi : (seg == nb) ? 2.0 * lo : 0.5 * (lo + hi);",
     "double s_ref = (seg == 0) ? 0.5 * hi : (seg == nb) ? 2.0 * lo : lo;"),
    ("ldlq_order_ascending", "while (j > 0 && H[perm[j - 1] * n + perm[j - 1]] < d) {",
     "while (j > 0 && H[perm[j - 1] * n + perm[j - 1]] > d) {"),
    ("ldlq_no_damping", "double lambda = n > 0 ? damp * (tr / (double)n) : 0.0;",
     "double lambda = 0.0 * damp * tr;"),
    ("ldlq_feedback_sign", "for (int64_t b = 0; b < a; ++b) x = x + e[b] * U[b * n + a];",
     "for (int64_t b = 0; b < a; ++b) x = x - e[b] * U[b * n + a];"),
    ("swiglu_exp_of_plus_g", "float e = nvfp4_ref_swiglu_exp(-g);", "float e = nvfp4_ref_swiglu_exp(g);"),
    ("swiglu_ln2_lo_dropped", "    r = fmaf(-n, ln2_lo, r);\n", "    r = fmaf(-n, 0.0f, r);\n"),
    ("swiglu_degree_5", "    float p = c[6];\n", "    float p = 0.0f;\n"),
    ("swiglu_bf16_truncates", "uint32_t r = b + 0x7FFFu + ((b >> 16) & 1u);", "uint32_t r = b;"),
    ("fp8_opt_ceil_not_taken", "if (nvfp4_ref_e4m3(cf) < s_opt && cf < E4M3_MAX_CODE) cc = cf + 1;",
     "if (nvfp4_ref_e4m3(cf) < s_opt && cf < E4M3_MAX_CODE) cc = cf;"),
]


PIN_FILES = ["tests/test_oracle_pins.py", "tests/test_oracle_bruteforce.py",
             "tests/test_oracle_subnormal.py", "tests/test_oracle_swiglu.py",
             "tests/test_oracle_windows.py", "tests/test_oracle_optimum.py",
             "tests/test_oracle_online.py", "tests/test_oracle_ldlq.py"]
PRIMARY_FILE = [("ldlq_", "tests/test_oracle_ldlq.py"),
                ("s_base_nearest", "tests/test_oracle_subnormal.py"),
                ("swiglu_", "tests/test_oracle_swiglu.py"),
                ("window_base_nearest", "tests/test_oracle_subnormal.py"),
                ("online_", "tests/test_oracle_online.py"),
                ("swizzle_", "tests/test_oracle_online.py"),
                ("norm_", "tests/test_oracle_online.py"),
                ("optimum_", "tests/test_oracle_optimum.py"),
                ("fp8_opt_", "tests/test_oracle_optimum.py"),
                ("tight_", "tests/test_oracle_windows.py"),
                ("window_clamp", "tests/test_oracle_windows.py"),
                ("window_offsets", "tests/test_oracle_windows.py")]


@pytest.mark.slow
@pytest.mark.parametrize("name,orig,planted", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, orig, planted, tmp_path):
    src = oracle.SRC.read_text()
    assert src.count(orig) == 1, f"anchor for {name} must occur exactly once"
    (tmp_path / "nvfp4_oracle.c").write_text(src.replace(orig, planted))
    (tmp_path / "nvfp4_oracle.h").write_text((oracle.HERE / "nvfp4_oracle.h").read_text())
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared", "-o",
                    str(lib), str(tmp_path / "nvfp4_oracle.c"), "-lm"], check=True)
    env = dict(os.environ, NVFP4_ORACLE_LIB=str(lib))
    # the whole pin suite, the file that pins the mutated function first (-x stops at the
    # first failure, so a caught mistake costs about one file)
    first = next((f for prefix, f in PRIMARY_FILE if name.startswith(prefix)), None)
    files = [f for f in PIN_FILES if f != first]
    if first:
        files.insert(0, first)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not slow", *files],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"planted mistake {name} was not caught:\n{r.stdout[-2000:]}"

"""Plant a plausible mistake in a copy of the oracle's C source and check that
the pins in test_oracle_pins.py catch it (CPU only).  The mutated library is
built in a temporary directory and loaded by a child pytest through
BNN_ORACLE_LIB; the committed oracle is never modified."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "bnn_oracle.c")

MUTATIONS = {
    "pad_zero_instead_of_minus_one":
        ("inside ? x[((n * H + hi) * W + wi) * C + c] : -1;",
         "inside ? x[((n * H + hi) * W + wi) * C + c] : 0;"),
    "sign_tie_to_plus_one":
        ("return v > 0.0f ?", "return v >= 0.0f ?"),
    "kernel_transposed":
        ("w[(((int64_t)f * KH + kh) * KW + kw) * C + c]",
         "w[(((int64_t)f * KH + kw) * KW + kh) * C + c]"),
    "kernel_mirrored_true_convolution":
        ("const int64_t hi = i * stride + kh - pad;\n      const int64_t wi = j * stride + kw - pad;\n      const int inside",
         "const int64_t hi = i * stride + (KH - 1 - kh) - pad;\n      const int64_t wi = j * stride + (KW - 1 - kw) - pad;\n      const int inside"),
    "stride_ignored":
        ("const int64_t hi = i * stride + kh - pad;\n      const int64_t wi = j * stride + kw - pad;\n      const int inside",
         "const int64_t hi = i + kh - pad;\n      const int64_t wi = j + kw - pad;\n      const int inside"),
    "dropped_last_kernel_column":
        ("for (int32_t kw = 0; kw < KW; ++kw) {\n      const int64_t hi",
         "for (int32_t kw = 0; kw < KW - 1; ++kw) {\n      const int64_t hi"),
    "threshold_strict":
        ("const int ge = S[p * F + f] >= thr[f];", "const int ge = S[p * F + f] > thr[f];"),
    "flip_dropped":
        ("const int bit = ge ^ (flip ? (flip[f] & 1) : 0);\n      out[p * F + f] = bit ? (int8_t)1 : (int8_t)-1;\n    }\n  }\n}\n\n/* The same threshold for real",
         "const int bit = ge;\n      out[p * F + f] = bit ? (int8_t)1 : (int8_t)-1;\n    }\n  }\n}\n\n/* The same threshold for real"),
    "pack_lsb_first":
        ("acc += (one_plus_x << (B - 1 - m)) >> 1;", "acc += (one_plus_x << m) >> 1;"),
    "pool_min":
        ("if (v > m) m = v;", "if (v < m) { m = v; } m = (int8_t)(m + 0 * v);"),
    "fc_sign_flipped":
        ("s += (int32_t)A[m * K + k] * B[n * K + k];", "s -= (int32_t)A[m * K + k] * B[n * K + k];"),
    "fconv_pad_minus_one":
        ("if (hi < 0 || hi >= H || wi < 0 || wi >= W) continue; /* 0.0 */",
         "if (hi < 0 || hi >= H || wi < 0 || wi >= W) { for (int32_t c = 0; c < C; ++c) s -= (double)w[((f * KH + kh) * (int64_t)KW + kw) * C + c]; continue; }"),
    "gray_red_blue_swapped":
        ("const float r = 0.299f * px[0];", "const float r = 0.299f * px[2];"),
    "gray_dropped_blue":
        ("return rg + b;", "return rg + 0.0f * b;"),
    "lbp_wrong_neighbour":
        ("static const int dc[3] = {-1, 1, -1};", "static const int dc[3] = {-1, 1, 1};"),
    "lbp_counterclockwise":
        ("static const int dr[3] = {-1, 0, 1};\n  static const int dc[3] = {-1, 1, -1};",
         "static const int dr[3] = {-1, 1, -1};\n  static const int dc[3] = {-1, 0, 1};"),
    "lbp_ties_exceed":
        ("if (g > centre) v = 1;", "if (g >= centre) v = 1;"),
    "lbp_outside_exceeds":
        ("          int8_t v = -1;\n          if (ni >= 0", "          int8_t v = 1;\n          if (ni >= 0"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor not found once: " + name
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                           "-ffp-contract=off", "-o", str(lib), str(mutated)])
    env = dict(os.environ, BNN_ORACLE_LIB=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 1, "pins did not catch mutation %s:\n%s" % (name, r.stdout[-2000:])

"""The pins must be able to fail: plant plausible mistakes in copies of the
oracle source (on the CPU, in a temporary directory) and check that the pin
suite rejects every one of them."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "gt_oracle.c")

MUTANTS = {
    "no_max_shift": ("const double w = exp(s[t] - m);", "const double w = exp(s[t]);"),
    "transposed_roles": (
        "elem(Q, dtype, (i * H + h) * (int64_t)D + d) *\n"
        "                           elem(K, dtype, (j * H + h) * (int64_t)D + d)",
        "elem(Q, dtype, (j * H + h) * (int64_t)D + d) *\n"
        "                           elem(K, dtype, (i * H + h) * (int64_t)D + d)"),
    "no_scale": ("s[t] = (double)scale * dot;", "s[t] = dot;"),
    "sign_flip": ("s[t] = (double)scale * dot;", "s[t] = -(double)scale * dot;"),
    "row_end_off_by_one": ("const int64_t deg = e - b;",
                           "const int64_t deg = e - b > 0 ? e - b - 1 : 0;"),
    "wrong_head_for_v": ("const double v = elem(V, dtype, (j * H + h) * (int64_t)D + d);",
                         "const double v = elem(V, dtype, (j * H + 0) * (int64_t)D + d);"),
    "lse_drops_max": ("lse[r * H + h] = m + log(Z);", "lse[r * H + h] = log(Z);"),
    "absagg_signed": ("if (a) a[d] += w * fabs(v);", "if (a) a[d] += w * v;"),
    "bf16_widening": ("uint32_t bits = (uint32_t)((const uint16_t*)base)[k] << 16;",
                      "uint32_t bits = (uint32_t)((const uint16_t*)base)[k] << 15;"),
    "bwd_drops_delta": ("const double ds = alpha * (da - delta);", "const double ds = alpha * da;"),
    "bwd_dkv_drops_delta": ("const double ds = alpha * (da - Dl[u * H + h]);",
                            "const double ds = alpha * da;"),
    "bwd_alpha_without_lse": ("const double alpha = exp(s[t] - L);", "const double alpha = exp(s[t]);"),
    "bwd_dk_without_scale": ("gk[d] += sc * ds * qv;", "gk[d] += ds * qv;"),
    "bwd_dv_without_alpha": ("gv[d] += alpha * go;", "gv[d] += go;"),
    "bwd_dq_sign": ("g[d] += sc * ds * kv;", "g[d] -= sc * ds * kv;"),
    "gatv2_slope_on_positive": ("(x > 0.0 ? x : sl * x)", "(x > 0.0 ? sl * x : x)"),
    "gatv2_no_attention_vector": ("acc += (double)att[h * D + d] * (x > 0.0 ? x : sl * x);",
                                  "acc += (x > 0.0 ? x : sl * x);"),
    "gatv2_left_as_value": ("const double v = elem(Rf, dtype, (j * H + h) * (int64_t)D + d);",
                            "const double v = elem(Lf, dtype, (j * H + h) * (int64_t)D + d);"),
    "gatv2_row_term_from_source": ("const double x = elem(Lf, dtype, (i * H + h) * (int64_t)D + d) +",
                                   "const double x = elem(Lf, dtype, (j * H + h) * (int64_t)D + d) +"),
    "reduce_tie_to_largest_source": ("better = k < best_key || (k == best_key && j < best_j);",
                                     "better = k < best_key || (k == best_key && j > best_j);"),
    "reduce_key_without_inversion": ("return (b & 0x80000000u) ? ~b : (b | 0x80000000u);",
                                     "return b | 0x80000000u;"),
    "reduce_key_ignores_sign_bit": ("return (b & 0x80000000u) ? ~b : (b | 0x80000000u);",
                                    "return b ^ 0x80000000u;"),
    "reduce_max_tie_to_largest": ("better = k > best_key || (k == best_key && j < best_j);",
                                  "better = k >= best_key;"),
    "reduce_empty_arg_zero": ("arg[r * F + f] = have ? best_j : -1;",
                              "arg[r * F + f] = have ? best_j : 0;"),
    "reduce_wrong_feature": ("const float x = (float)elem(X, dtype, (int64_t)j * F + f);",
                             "const float x = (float)elem(X, dtype, (int64_t)j * F);"),
}
PIN_FILES = ["test_oracle_pins.py", "test_oracle_bwd_pins.py", "test_oracle_gatv2_pins.py",
             "test_oracle_reduce_pins.py"]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    src = open(SRC).read()
    old, new = MUTANTS[name]
    assert old in src, "mutation site moved: update the mutant table"
    csrc = tmp_path / "gt_oracle.c"
    csrc.write_text(src.replace(old, new))
    so = tmp_path / "libgt_oracle.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", str(csrc), "-o",
                    str(so), "-lm"], check=True)
    files = [os.path.join(ROOT, "tests", f) for f in PIN_FILES]
    code = ("import sys, oracle, pytest; oracle._SO = %r; "
            "sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider'] + %r))"
            % (str(so), files))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                       env=dict(os.environ, OMP_NUM_THREADS="2"))
    assert r.returncode != 0, "pins accepted a planted mistake: " + name

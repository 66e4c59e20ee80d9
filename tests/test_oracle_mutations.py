"""The oracle's pins catch plausible mistakes.

Each case plants one mistake into a copy of the oracle source (on the CPU,
in a temporary directory), builds it, and runs the pin suites against the
mutated library; at least one pin must fail.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "np_oracle.c")
PINS = ["tests/test_oracle_encoding.py", "tests/test_oracle_predict.py",
        "tests/test_oracle_select.py", "tests/test_oracle_delta.py",
        "tests/test_oracle_mlp.py", "tests/test_oracle_centroid.py",
        "tests/test_oracle_swiglu.py"]

MUTATIONS = {
    # predictor: transposed / shifted A operand
    "predict_A_transposed":
        ("acc += orc_load(wdtype, A, row + c) * hv[c];",
         "acc += orc_load(wdtype, A, (size_t)l * r * d + (size_t)c * r + j) * hv[c];"),
    "predict_z_dropped_term":
        ("for (int j = 0; j < r; ++j) acc += orc_load(wdtype, B, row + j) * z[j];",
         "for (int j = 1; j < r; ++j) acc += orc_load(wdtype, B, row + j) * z[j];"),
    # selection: ties to the larger id
    "select_tie_to_larger_id":
        ("return a < b ? -1 : (a > b ? 1 : 0);\n}\n\nstatic int by_int_asc",
         "return a > b ? -1 : (a < b ? 1 : 0);\n}\n\nstatic int by_int_asc"),
    # delta: most-recently-used eviction
    "delta_mru_eviction":
        ("if (ua != ub) return ua < ub ? -1 : 1;", "if (ua != ub) return ua > ub ? -1 : 1;"),
    # delta: victims' slots appended unsorted
    "delta_pool_unsorted":
        ("qsort(pool, (size_t)npool, sizeof(int32_t), by_int_asc);", ""),
    # delta: last_used not refreshed for hits
    "delta_lastused_only_incoming":
        ("for (int j = 0; j < na; ++j) U[A[j]] = t;", "for (int j = 0; j < ni; ++j) U[I[j]] = t;"),
    # MLP: ReLU dropped, wrong row for down^T
    "mlp_no_relu":
        ("return (g > 0.0 ? g : 0.0) * u;", "return g * u;"),
    # SwiGLU: sigmoid of -g; eq. 1 zeroing a magnitude equal to T
    "silu_exp_sign":
        ("return g / (1.0 + exp(-g)) * u;", "return g / (1.0 + exp(g)) * u;"),
    "eq1_drops_equal_magnitude":
        ("return fabs(a) < thr ? 0.0 : a;", "return fabs(a) <= thr ? 0.0 : a;"),
    # percentile: the (m+1)-th smallest; thresholded set strictly above T
    "percentile_off_by_one":
        ("out[r] = mag[m - 1];", "out[r] = mag[m < n ? m : m - 1];"),
    "threshold_active_strict":
        ("if (fabsf(v) >= thr[r]) {", "if (fabsf(v) > thr[r]) {"),
    "mlp_down_reads_up_row":
        ("acc[c] += a * orc_load(wdtype, storage, base + 2 * (size_t)d + c);",
         "acc[c] += a * orc_load(wdtype, storage, base + (size_t)d + c);"),
    # rounding: ties away from zero
    # centroid predictor: tie to the last maximum, union instead of intersection
    "centroid_tie_to_last":
        ("if (lg[c] > lg[best]) best = c;", "if (lg[c] >= lg[best]) best = c;"),
    "centroid_union":
        ("uint32_t m = g[w] & u[w];", "uint32_t m = g[w] | u[w];"),
    # off by one in the active-slot list of a variable-size set
    "delta_active_slots_off_by_one":
        ("for (int j = 0; j < na; ++j) AS[j] = P[A[j]];",
         "for (int j = 0; j + 1 < na; ++j) AS[j] = P[A[j]];"),
    "round_ties_away":
        ("if (frac > 0.5 || (frac == 0.5 && fmod(lo, 2.0) != 0.0)) r = lo + 1.0;",
         "if (frac >= 0.5) r = lo + 1.0;"),
    # binary16 decoding: wrong exponent bias
    "f16_bias_off_by_one":
        ("v = ldexp((double)(1024 + f), e - 25);", "v = ldexp((double)(1024 + f), e - 24);"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = tmp_path / "np_oracle_mut.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mut.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", str(lib),
                           str(mutated), "-lm"])
    env = dict(os.environ, NP_ORACLE_LIB_OVERRIDE=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *PINS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"no pin failed for planted mistake {name}:\n{r.stdout[-2000:]}"

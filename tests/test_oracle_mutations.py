"""The oracle's pins must catch plausible slips in the oracle itself.

Each case plants one mistake in a copy of the oracle's C source (CPU only),
builds it, and runs the pin suite against it; the suite must fail.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "logra_oracle.c")

MUTATIONS = {
    "transposed_G_layout": ("gb[(int64_t)o * k_in + i] += dp[o] * xp[i]",
                            "gb[(int64_t)i * k_out + o] += dp[o] * xp[i]"),
    "mask_ignored": ("if (mask && mask[bt] == 0) continue; /* masked: never read */", ""),
    "mask_multiply_not_select": ("if (mask && mask[bt] == 0) continue; /* masked: never read */",
                                 "double mm = mask ? (double)mask[bt] : 1.0;"),
    "mean_not_sum_over_tokens": ("gb[(int64_t)o * k_in + i] += dp[o] * xp[i];",
                                 "gb[(int64_t)o * k_in + i] += dp[o] * xp[i] / (double)T;"),
    "cov_missing_term": ("for (int b = 0; b < B; ++b)\n                s += widen(g",
                         "for (int b = 1; b < B; ++b)\n                s += widen(g"),
    "damping_uses_D_minus_1": ("double lambda = r * tr / (double)D;",
                               "double lambda = r * tr / (double)(D - 1);"),
    "damping_unnormalised_S": ("tr += S[(int64_t)d * D + d] / (double)N;",
                               "tr += S[(int64_t)d * D + d];"),
    "backsolve_wrong_index": ("s -= L[(int64_t)m * D + i] * z[m];",
                              "s -= L[(int64_t)i * D + m] * z[m];"),
    "scores_sign": ("acc += widen(te", "acc -= widen(te"),
    "topk_ties_to_higher_index": ("return ia < ib;", "return ia > ib;"),
    "bf16_widen_wrong_shift": ("<< 16;", "<< 15;"),
    "self_influence_drops_damping": ("const int rc = oracle_precondition(S, D, N, r, g, g_dtype, ld_g, rows, y, D, NULL);",
                                     "const int rc = oracle_precondition(S, D, N, r > 0 ? 1e-12 : r, g, g_dtype, ld_g, rows, y, D, NULL);"),
    "normalise_without_sqrt": ("? s[(int64_t)q * ld_s + j] / sqrt(den) : 0.0;",
                               "? s[(int64_t)q * ld_s + j] / den : 0.0;"),
    "act_cov_mask_ignored": ("if (mask && mask[bt] == 0) continue;\n                double ai",
                             "double ai"),
    "act_cov_skips_first_token": ("for (int t = 0; t < T; ++t) {\n                int64_t bt = (int64_t)b * T + t;\n                if (mask && mask[bt] == 0) continue;\n                double ai",
                                  "for (int t = 1; t < T; ++t) {\n                int64_t bt = (int64_t)b * T + t;\n                if (mask && mask[bt] == 0) continue;\n                double ai"),
}

# Slips in the numpy part of the oracle (the PCA initialisation), planted in a
# copy of the oracle package that the pin suite imports in place of the real one.
PY_SRC = os.path.join(ROOT, "oracle", "__init__.py")
PY_MUTATIONS = {
    "pca_bottom_k": ('order = np.argsort(-w, kind="stable")[:k]', 'order = np.argsort(w, kind="stable")[:k]'),
    "pca_columns_as_rows": ("P = V[:, order].T.copy()", "P = V[order, :].copy()"),
    "pca_no_sign_rule": ("if P[r, i] < 0:", "if False:"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert old in src, f"mutation anchor not found: {name}"
    src = src.replace(old, new, 1)
    if name == "mask_multiply_not_select":
        # a multiply-by-mask version: reads masked tokens and scales them by 0
        src = src.replace("gb[(int64_t)o * k_in + i] += dp[o] * xp[i];",
                          "gb[(int64_t)o * k_in + i] += mm * dp[o] * xp[i];", 1)
    with tempfile.TemporaryDirectory() as td:
        c = os.path.join(td, "m.c")
        so = os.path.join(td, "m.so")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared", c, "-o", so, "-lm"],
                       check=True)
        env = dict(os.environ, LOGRA_ORACLE_LIB=so)
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                           env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
        assert r.returncode != 0, f"pins did not catch mutation {name}:\n{r.stdout[-2000:]}"


@pytest.mark.parametrize("name", sorted(PY_MUTATIONS))
def test_pins_catch_python_mutation(name):
    old, new = PY_MUTATIONS[name]
    src = open(PY_SRC).read()
    assert old in src, f"mutation anchor not found: {name}"
    with tempfile.TemporaryDirectory() as td:
        pkg = os.path.join(td, "oracle")
        os.makedirs(pkg)
        open(os.path.join(pkg, "__init__.py"), "w").write(src.replace(old, new, 1))
        driver = (
            "import importlib.util, sys\n"
            f"spec = importlib.util.spec_from_file_location('oracle', {os.path.join(pkg, '__init__.py')!r}, "
            f"submodule_search_locations=[{pkg!r}])\n"
            "m = importlib.util.module_from_spec(spec); sys.modules['oracle'] = m; spec.loader.exec_module(m)\n"
            "import pytest\n"
            f"sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', {os.path.join(ROOT, 'tests', 'test_oracle_pins.py')!r}]))\n")
        import oracle
        env = dict(os.environ, LOGRA_ORACLE_LIB=oracle.build(force=False))
        r = subprocess.run([sys.executable, "-c", driver], env=env, cwd=ROOT, capture_output=True, text=True,
                           timeout=300)
        assert r.returncode != 0, f"pins did not catch mutation {name}:\n{r.stdout[-2000:]}"

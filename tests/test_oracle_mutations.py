"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a dropped
term, a flipped sign, a wrong index or tie-break, a transposed operand),
builds it on the CPU, and runs the pin suite against it in a subprocess: every
mutant must make at least one pin fail.  The real oracle is never modified.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "drop-derivative": ("b = b + dterm;", "(void)dterm;"),
    "gate-sign": ("(e_prev[i] > 0.0f && de > 0.0f)", "(e_prev[i] > 0.0f && de < 0.0f)"),
    "drop-integral": ("float b = bias[i] + u;", "float b = bias[i] + 0.0f * u;"),
    "no-centering": ("if (center) {", "if (0) {"),
    "error-sign": ("int64_t num = S - (int64_t)E * (int64_t)counts[i];",
                   "int64_t num = (int64_t)E * (int64_t)counts[i] - S;"),
    "tie-break-highest": ("return ia < ib;", "return ia > ib;"),
    "bias-in-gate-weights": ("den = den + s[idx[r]];", "den = den + s[idx[r]] + bias[idx[r]];"),
    "transposed-weight": ("load_elem(W, dtype, (int64_t)i * d + k)", "load_elem(W, dtype, (int64_t)k * d + i)"),
    "sigmoid-sign": ("exp(-z)", "exp(z)"),
    "maxvio-uses-min": ("(int64_t)E * mx - S", "(int64_t)E * mn - S"),
    "mean-over-P": ("tree_sum(bt, E) / (float)E", "tree_sum(bt, E) / (float)(E + 1)"),
    "diag-m-floor": ("const int32_t m = (E + 9) / 10;", "const int32_t m = E / 10;"),
    "diag-gate-new-eprev": ("float de = e - ep_old[i];", "float de = e - e_prev[i];"),
    "entropy-log2": ("if (x > 0.0) h -= x * log(x);", "if (x > 0.0) h -= x * log2(x);"),
    "full-entropy-unclamped": ("if (v > 0.0f) C += (double)v;", "C += (double)v;"),
    "qb-alpha-kth": ("for (int32_t r = 0; r <= K; ++r) {", "for (int32_t r = 0; r < K; ++r) {"),
    "qb-quantile-level": ("const int64_t k = (T * (int64_t)(E - K) + E - 1) / E;",
                          "const int64_t k = (T * (int64_t)K + E - 1) / E;"),
    "qb-floor": ("const int64_t k = (T * (int64_t)(E - K) + E - 1) / E;",
                 "const int64_t k = (T * (int64_t)(E - K)) / E;"),
    "qb-no-negation": ("const float Q = -q;", "const float Q = q;"),
    "qb-ema-weights": ("const float take = (1.0f - rho) * Q;", "const float take = rho * Q;"),
    "qb-biased-margin": ("d[t] = (s[t * (int64_t)E + j] - alpha[t]) + 0.0f;",
                         "d[t] = (s[t * (int64_t)E + j] + bias[j] - alpha[t]) + 0.0f;"),
    "aux-no-max-shift": ("pt[i] = exp(zt[i] - m);", "pt[i] = exp(zt[i]);"),
    "aux-unnormalised-p": ("for (int32_t i = 0; i < E; ++i) pt[i] = pt[i] / Z;", "(void)Z;"),
    "aux-raw-gate-weights": ("(float)(pt[it[r]] / den)", "(float)pt[it[r]]"),
    "aux-f-over-tk": ("f[i] = (double)counts[i] / (double)T;", "f[i] = (double)counts[i] / (double)(T * K);"),
    "aux-loss-misaligned": ("L = L + f[i] * P[i];", "L = L + f[i] * P[E - 1 - i];"),
    "aux-rank-ascending": ("const float v = (float)zt[i];", "const float v = -(float)zt[i];"),
    "softmax-entropy-no-max-shift": ("for (int32_t e = 0; e < E; ++e) Z += exp((double)zt[e] - m);",
                                     "for (int32_t e = 0; e < E; ++e) Z += exp((double)zt[e]);"),
    "softmax-entropy-log2": ("if (p > 0.0) h -= p * log(p);", "if (p > 0.0) h -= p * log2(p);"),
    "softmax-entropy-sum-over-tokens": ("    return acc / (double)T;\n}\n\n/* S1", "    return acc;\n}\n\n/* S1"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    src = open(oracle.SRC_PATH).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation anchor missing: {old}"
    csrc = tmp_path / "mutant.c"
    csrc.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    cmd = [c if c not in (oracle.LIB_PATH, oracle.SRC_PATH) else (str(lib) if c == oracle.LIB_PATH else str(csrc))
           for c in oracle.BUILD_CMD]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, IDB_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} passed every pin:\n{r.stdout[-2000:]}"

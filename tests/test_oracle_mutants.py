"""The oracle's pins catch plausible mistakes (mutation test, CPU only).

Each mutant is the oracle's C source with one plausible slip planted in a
copy: a flipped sign, a dropped term or factor, the wrong EMA state, a
missing mask, truncating instead of rounding, and so on.  The mutant is
built with the oracle's own flags and the pin suites (tests/test_oracle_pins.py
and tests/test_oracle_decide_gram.py, unchanged) are run against it; every
mutant must make at least one pin fail.  A mutant replaces every occurrence
of its text, and states how many there are (the step and the decision from a
Gram matrix share some statements).  The committed oracle is never modified.
"""
import concurrent.futures
import os
import subprocess
import sys


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCE = os.path.join(ROOT, "oracle", "edit_oracle.c")
sys.path.insert(0, ROOT)
from oracle.build import CFLAGS  # noqa: E402

PIN_FILES = ["test_oracle_pins.py", "test_oracle_decide_gram.py"]

# (name, text in the source, replacement[, occurrences])
MUTANTS = [
    ("delta sign", "return r - (double)theta[i];", "return (double)theta[i] - r;"),
    ("norm without sqrt", "return sqrt(s);", "return s;"),
    ("z-test direction", "double lhs = G - mu;", "double lhs = mu - G;"),
    ("z-test on variance", "double rhs = delta * sigma;", "double rhs = delta * sigma * sigma;"),
    ("EMA weights swapped", "double mu_new = alpha * G + (1.0 - alpha) * (*mu);",
     "double mu_new = (1.0 - alpha) * G + alpha * (*mu);"),
    ("sigma from the old mean", "double dev = G - mu_new;", "double dev = G - *mu;"),
    ("sigma decay dropped", "sqrt((1.0 - alpha) * (*sigma) * (*sigma) + alpha * dev * dev)",
     "sqrt((*sigma) * (*sigma) + alpha * dev * dev)"),
    ("no warm-up", "const int z_test = ae && ema->round >= cfg->warmup_rounds;",
     "const int z_test = ae;"),
    ("non-finite not masked", "anomalous[j] = !isfinite(G[j]);", "anomalous[j] = 0;"),
    ("EMA updated for flagged workers", "if (!anomalous[j]) ema_update(", "if (1) ema_update("),
    ("no rollback", "if (n_ok == 0) {", "if (n_ok < 0) {", 2),
    ("softmax of +G", "exp(-(G[j] - g0))", "exp((G[j] - g0))"),
    ("weights not normalised", "for (int j = 0; j < K; ++j) w[j] /= gamma;", ""),
    ("uniform weight over all K", "1.0 / (double)n_ok;", "1.0 / (double)K;"),
    ("flagged workers averaged", "if (!anomalous[j]) s += w[j] *", "s += w[j] *"),
    ("clip without the cap", "fmin(cfg->clip_threshold / (gbar + cfg->clip_eps), 1.0)",
     "cfg->clip_threshold / (gbar + cfg->clip_eps)"),
    ("clip epsilon misplaced", "cfg->clip_threshold / (gbar + cfg->clip_eps)",
     "(cfg->clip_threshold / gbar + cfg->clip_eps)"),
    ("momentum sign", "double b_new = rho * (double)momentum[i] + g;",
     "double b_new = rho * (double)momentum[i] - g;"),
    ("heavy ball instead of Nesterov", "nu * (g + rho * b_new)", "nu * b_new"),
    ("Nesterov look-ahead without rho", "nu * (g + rho * b_new)", "nu * (g + b_new)"),
    ("last bf16 replica not written", "for (int j = 0; j < K; ++j) ((uint16_t *)replicas[j])[i] = h;",
     "for (int j = 0; j + 1 < K; ++j) ((uint16_t *)replicas[j])[i] = h;"),
    ("bf16 truncated", "if (toward_zero == bits) return (uint16_t)(bits >> 16);",
     "return (uint16_t)(bits >> 16);"),
    ("bf16 ties to odd", "return ((toward_zero >> 16) & 1u) ? (uint16_t)(away >> 16)",
     "return ((toward_zero >> 16) & 1u) == 0 ? (uint16_t)(away >> 16)"),
    # the decision from a given Gram matrix
    ("Gram norm without sqrt", "G[j] = sqrt(GRAM_AT(j, j));", "G[j] = GRAM_AT(j, j);"),
    ("Gbar from the diagonal only", "q += w[j] * w[k] * (j <= k ? GRAM_AT(j, k) : GRAM_AT(k, j));",
     "if (j == k) q += w[j] * w[k] * GRAM_AT(j, j);"),
    ("Gbar with w_j squared", "q += w[j] * w[k] *", "q += w[j] * w[j] *"),
    ("triangular index off by one", "gram[(j) * K - ((j) * ((j) - 1)) / 2 + ((k) - (j))]",
     "gram[(j) * K - ((j) * ((j) + 1)) / 2 + ((k) - (j))]"),
    ("flagged worker kept in Gbar", "if (anomalous[k]) continue;", ""),
    ("negative squared norm not clamped", "sqrt(q > 0.0 ? q : 0.0)", "sqrt(q)"),
    ("round not advanced by the Gram decision", "r.clip_coef = clip_coefficient(cfg, gbar);\n\n  ema->round += 1;",
     "r.clip_coef = clip_coefficient(cfg, gbar);\n"),
]


def _build_and_pin(tmp_path, i, name, old, new, count=1):
    src = open(SOURCE).read()
    assert src.count(old) == count, f"{name}: the text to mutate must occur {count} time(s)"
    c = tmp_path / f"mutant{i}.c"
    so = tmp_path / f"mutant{i}.so"
    c.write_text(src.replace(old, new))
    subprocess.run(["gcc", *CFLAGS, "-I", os.path.join(ROOT, "oracle"), "-o", str(so), str(c), "-lm"],
                   check=True, capture_output=True)
    env = dict(os.environ, EDIT_ORACLE_LIBRARY=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *[os.path.join(ROOT, "tests", f) for f in PIN_FILES]],
                       capture_output=True, text=True, env=env, timeout=300, cwd=ROOT)
    failed = [ln for ln in r.stdout.splitlines() if ln.startswith("FAILED")]
    return name, r.returncode, failed[:1]


def test_every_mutant_fails_a_pin(tmp_path):
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        results = list(ex.map(lambda a: _build_and_pin(tmp_path, a[0], *a[1]), enumerate(MUTANTS)))
    survivors = [name for name, rc, _ in results if rc == 0]
    report = "\n".join(f"{name}: rc={rc} {failed}" for name, rc, failed in results)
    print(report)
    assert not survivors, f"mutants not caught by any pin: {survivors}"

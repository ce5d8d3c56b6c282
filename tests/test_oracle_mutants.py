"""The oracle's pins must catch plausible mistakes in it.

Each case below is one slip a careful reader could make while writing the
oracle from the paper: a dropped term, a wrong sign, the wrong momentum, a
transposed operand, an update out of order.  The case applies it to a copy
of the oracle source, builds the copy with the oracle's own compiler flags,
and runs the pin tests against it (through RIKFAD_ORACLE_LIB).  Every
mutant must make a pin fail.  The oracle source itself stays untouched,
and nothing here runs on a GPU.
"""
import concurrent.futures
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")

RIKFAD_PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")
ADAFM_PINS = os.path.join(ROOT, "tests", "test_adafm_oracle.py")

# (name, source file, text as written, mistaken text, pin file)
MUTANTS = [
    # B and A (Table rows B, A)
    ("drift_with_p_n", "rikfad_oracle.c",
     "const double xu = x[e] + h * pb[e];", "const double xu = x[e] + h * p[e];", RIKFAD_PINS),
    ("kick_sign", "rikfad_oracle.c",
     "pb[e] = p[e] - h * g[e];", "pb[e] = p[e] + h * g[e];", RIKFAD_PINS),
    # C: which momentum drives the factors, and their filter
    ("row_sums_of_p_b", "rikfad_oracle.c",
     "for (int64_t j = 0; j < n; ++j) s += p1[i * n + j] * p1[i * n + j];",
     "for (int64_t j = 0; j < n; ++j) s += pb[i * n + j] * pb[i * n + j];", RIKFAD_PINS),
    ("column_sums_of_p_b", "rikfad_oracle.c",
     "colsq[j] += p1[i * n + j] * p1[i * n + j];",
     "colsq[j] += pb[i * n + j] * pb[i * n + j];", RIKFAD_PINS),
    ("rows_take_column_sums", "rikfad_oracle.c",
     "r[i] = a * r[i] + kappa * rowsq[i];", "r[i] = a * r[i] + kappa * colsq[i % n];",
     RIKFAD_PINS),
    ("gain_without_1_over_mu", "rikfad_oracle.c",
     "(-expm1(-ah)) / (hp->mu * hp->alpha)", "(-expm1(-ah)) / (hp->alpha)", RIKFAD_PINS),
    ("factors_without_decay", "rikfad_oracle.c",
     "out[0] = exp(-ah);", "out[0] = 1.0;", RIKFAD_PINS),
    ("alpha_zero_limit_without_mu", "rikfad_oracle.c",
     ": hp->h / hp->mu;", ": hp->h;", RIKFAD_PINS),
    # eq. (xi_def)
    ("eps_in_numerator", "rikfad_oracle.c",
     "(r[i] * c[j]) / denom", "(r[i] * c[j] + eps_stab) / denom", RIKFAD_PINS),
    ("eps_dropped", "rikfad_oracle.c",
     "const double denom = s + eps_stab;", "const double denom = s + 0.0 * eps_stab;",
     RIKFAD_PINS),
    ("zero_denominator_unguarded", "rikfad_oracle.c",
     "(denom == 0.0) ? 0.0 : (r[i] * c[j]) / denom", "(r[i] * c[j]) / denom", RIKFAD_PINS),
    ("denominator_from_columns", "rikfad_oracle.c",
     "for (int64_t i = 0; i < m; ++i) s += r[i];",
     "for (int64_t j = 0; j < n; ++j) s += c[j];", RIKFAD_PINS),
    # C: half-kicks
    ("full_kick_not_half", "rikfad_oracle.c",
     "p1[e] = pb[e] * exp(-0.5 * h * xi[e]);", "p1[e] = pb[e] * exp(-h * xi[e]);",
     RIKFAD_PINS),
    ("second_half_kick_with_old_factors", "rikfad_oracle.c",
     "    orc_rank1_friction(m, n, r, c, hp->eps_stab, xi);\n"
     "    for (int64_t e = 0; e < k; ++e) {\n        const double p2",
     "    for (int64_t e = 0; e < k; ++e) {\n        const double p2", RIKFAD_PINS),
    # D
    ("no_damping", "rikfad_oracle.c",
     "        p[e] = p2 * d;\n    }\n\n    free(pb); free(p1);",
     "        p[e] = p2;\n    }\n\n    free(pb); free(p1);", RIKFAD_PINS),
    # element-wise iKFAD (vectors)
    ("vector_friction_of_p_b", "rikfad_oracle.c",
     "xi[e] = a * xi[e] + kappa * (p1 * p1);", "xi[e] = a * xi[e] + kappa * (pb[e] * pb[e]);",
     RIKFAD_PINS),
    ("vector_second_half_kick_before_update", "rikfad_oracle.c",
     "        xi[e] = a * xi[e] + kappa * (p1 * p1);\n"
     "        const double p2 = p1 * exp(-0.5 * h * xi[e]);",
     "        const double p2 = p1 * exp(-0.5 * h * xi[e]);\n"
     "        xi[e] = a * xi[e] + kappa * (p1 * p1);", RIKFAD_PINS),
    # storage
    ("bf16_truncates", "rikfad_oracle.c",
     "nearbyint(ldexp(av, -qexp))", "trunc(ldexp(av, -qexp))", RIKFAD_PINS),
    ("vectors_take_the_rank1_path", "rikfad_oracle.c",
     "if (T->m == 1 || T->n == 1) {", "if (0) {", RIKFAD_PINS),
    # Adafactor-m baseline
    ("adafm_beta2_off_by_one", "adafm_oracle.c",
     "return 1.0 - pow((double)t, decay_rate);", "return 1.0 - pow((double)t + 1.0, decay_rate);",
     ADAFM_PINS),
    ("adafm_eps1_dropped", "adafm_oracle.c",
     "q[e] = g[e] * g[e] + hp->eps1;", "q[e] = g[e] * g[e];", ADAFM_PINS),
    ("adafm_second_moment_without_sum", "adafm_oracle.c",
     "(r[i] * c[j]) / sr", "(r[i] * c[j])", ADAFM_PINS),
    ("adafm_update_without_sqrt", "adafm_oracle.c",
     "for (int64_t e = 0; e < k; ++e) u[e] = (v[e] == 0.0) ? 0.0 : g[e] / sqrt(v[e]);",
     "for (int64_t e = 0; e < k; ++e) u[e] = (v[e] == 0.0) ? 0.0 : g[e] / v[e];", ADAFM_PINS),
    ("adafm_clip_ignores_threshold", "adafm_oracle.c",
     "div = rms / hp->clip_threshold;", "div = rms;", ADAFM_PINS),
    ("adafm_momentum_without_1_minus_beta1", "adafm_oracle.c",
     "(1.0 - hp->beta1) * (a * uhat)", "(a * uhat)", ADAFM_PINS),
    ("adafm_parameter_moves_up", "adafm_oracle.c",
     "const double xu = x[e] - mom[e];", "const double xu = x[e] + mom[e];", ADAFM_PINS),
    ("adafm_factor_weights_swapped", "adafm_oracle.c",
     "r[i] = b * r[i] + (1.0 - b) * s;", "r[i] = (1.0 - b) * r[i] + b * s;", ADAFM_PINS),
    ("adafm_scale_floor_dropped", "adafm_oracle.c",
     "(rms > hp->eps2 ? rms : hp->eps2)", "rms", ADAFM_PINS),
]


def _build(workdir, fname, old, new):
    """Copy the oracle sources to workdir, apply the mistake, build."""
    for f in ("rikfad_oracle.c", "rikfad_oracle.h", "adafm_oracle.c", "adafm_oracle.h"):
        shutil.copy(os.path.join(ORACLE, f), workdir)
    path = os.path.join(workdir, fname)
    with open(path) as fh:
        src = fh.read()
    assert src.count(old) == 1, f"mutation anchor not unique in {fname}: {old!r}"
    with open(path, "w") as fh:
        fh.write(src.replace(old, new))
    lib = os.path.join(workdir, "liboracle_mutant.so")
    # the oracle's own flags (oracle/build.py)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
                    "-ffp-contract=off", "-w",
                    os.path.join(workdir, "rikfad_oracle.c"),
                    os.path.join(workdir, "adafm_oracle.c"), "-o", lib, "-lm"], check=True)
    return lib


def _run_pins(lib, pins):
    env = dict(os.environ, RIKFAD_ORACLE_LIB=lib, OMP_NUM_THREADS="1")
    out = subprocess.run([sys.executable, "-m", "pytest", pins, "-x", "-q", "-p",
                          "no:cacheprovider", "-W", "ignore"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return out.returncode, out.stdout[-2000:]


def test_unmutated_copy_passes_the_pins(tmp_path):
    """The harness itself: an unchanged copy built the same way passes."""
    lib = _build(str(tmp_path), "rikfad_oracle.c", "int orc_coefficients(",
                 "int orc_coefficients(")
    for pins in (RIKFAD_PINS, ADAFM_PINS):
        rc, out = _run_pins(lib, pins)
        assert rc == 0, out


def test_every_mutant_fails_a_pin(tmp_path):
    def one(case):
        name, fname, old, new, pins = case
        work = tmp_path / name
        work.mkdir()
        lib = _build(str(work), fname, old, new)
        rc, out = _run_pins(lib, pins)
        return name, rc, out

    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(one, MUTANTS))
    survivors = [(name, out) for name, rc, out in results if rc != 1]
    assert not survivors, "mutants not caught (pytest exit status != 1):\n" + "\n\n".join(
        f"{name}:\n{out}" for name, out in survivors)

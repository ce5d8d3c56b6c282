"""The fp64 oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle's C sources are built with its own flags (oracle/build.py) plus
-fsanitize=address,undefined, and its pin tests (test_oracle_pins.py,
test_adafm_oracle.py) run against that build through RIKFAD_ORACLE_LIB, so
an out-of-bounds access, a use after free or undefined behaviour anywhere
the pins drive the oracle aborts the run.  The sanitizer runtime is
preloaded ahead of whatever the environment already preloads (the Python
interpreter itself is not instrumented; leak checking is off for it).
CPU only."""
import concurrent.futures
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
PINS = [os.path.join(ROOT, "tests", "test_oracle_pins.py"),
        os.path.join(ROOT, "tests", "test_adafm_oracle.py")]


def _asan_runtime():
    out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                         check=True)
    return out.stdout.strip()


def test_oracle_pins_pass_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liboracle_sanitized.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fno-omit-frame-pointer",
                    os.path.join(ORACLE, "rikfad_oracle.c"), os.path.join(ORACLE, "adafm_oracle.c"),
                    "-o", lib, "-lm"], check=True)
    # the build really is instrumented
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms

    asan = _asan_runtime()
    assert os.path.exists(asan), asan
    prior = os.environ.get("LD_PRELOAD")
    env = dict(os.environ, RIKFAD_ORACLE_LIB=lib, OMP_NUM_THREADS="2",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1",
               LD_PRELOAD=asan + (":" + prior if prior else ""))

    def run(pins):
        out = subprocess.run([sys.executable, "-m", "pytest", pins, "-x", "-q", "-p",
                              "no:cacheprovider", "-W", "ignore"],
                             cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
        return pins, out.returncode, out.stdout[-3000:] + out.stderr[-3000:]

    with concurrent.futures.ThreadPoolExecutor(len(PINS)) as ex:
        results = list(ex.map(run, PINS))
    bad = [(p, out) for p, rc, out in results if rc != 0]
    assert not bad, "\n\n".join(f"{p}:\n{out}" for p, out in bad)
    for _, _, out in results:
        assert "passed" in out and "runtime error" not in out

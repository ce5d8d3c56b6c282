"""Build step for the fp64 oracle library (test infrastructure).

Compiles ``rikfad_oracle.c`` (R-iKFAD, iKFAD) and ``adafm_oracle.c``
(Adafactor-m) with gcc into ``liboracle_rikfad.so`` beside them.
IEEE semantics are kept: no fast-math and no floating-point contraction, so
every operation is the fp64 operation the source writes.
"""
import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose=False):
    srcs = [os.path.join(_HERE, f) for f in ("rikfad_oracle.c", "adafm_oracle.c")]
    out = os.path.join(_HERE, "liboracle_rikfad.so")
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
           *srcs, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

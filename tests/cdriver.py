"""Build of tests/c_abi_step.c, the plain C program that drives the library
through include/rikfad.h alone and checks it against the fp64 oracle
(test infrastructure: it links the oracle)."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi_step.c")
OUT_DIR = os.path.join(ROOT, "tests", "_bin")
OUT = os.path.join(OUT_DIR, "c_abi_step")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
LIB_DIR = os.path.join(ROOT, "paper_2609_30342_amd")
ORACLE_DIR = os.path.join(ROOT, "oracle")


def build():
    """Compile the driver with gcc as C11 (host code only) if it is missing
    or older than its source or the libraries; returns its path."""
    deps = [SRC, os.path.join(ROOT, "include", "rikfad.h"),
            os.path.join(LIB_DIR, "librikfad.so"),
            os.path.join(ORACLE_DIR, "liboracle_rikfad.so")]
    for d in deps[2:]:
        if not os.path.exists(d):
            raise FileNotFoundError(f"{d} is not built")
    if os.path.exists(OUT) and os.path.getmtime(OUT) >= max(os.path.getmtime(d) for d in deps):
        return OUT
    os.makedirs(OUT_DIR, exist_ok=True)
    tmp = OUT + f".tmp{os.getpid()}"
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{ORACLE_DIR}", SRC, "-o", tmp,
           f"-L{LIB_DIR}", "-lrikfad", f"-L{ORACLE_DIR}", "-loracle_rikfad",
           f"-L{ROCM}/lib", "-lamdhip64", "-lm",
           f"-Wl,-rpath,{LIB_DIR}:{ORACLE_DIR}:{ROCM}/lib"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    return OUT

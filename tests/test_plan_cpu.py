"""The tile and finalisation tables against the kernels' index arithmetic,
replayed on the CPU (tests/plan_check.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer: in-bounds accesses, every element updated once,
every partial sum written once, disjoint workspace regions."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_plan_tables_match_kernel_indexing(tmp_path):
    exe = tmp_path / "plan_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                    f"-I{ROOT}", os.path.join(ROOT, "tests", "plan_check.cpp"),
                    os.path.join(ROOT, "paper_2609_30342_amd", "csrc", "plan.cpp"),
                    "-o", str(exe)], check=True)
    out = subprocess.run([str(exe), "60"], capture_output=True, text=True, timeout=600)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "0 failures" in out.stdout

"""The library driven from plain C (tests/c_abi_step.c): a C11 program that
includes include/rikfad.h, allocates with the HIP runtime, calls
rikfad_create / rikfad_step / rikfad_sync_momentum / rikfad_nonfinite /
rikfad_destroy, and checks every tensor against the fp64 oracle itself.  No
Python binding and no PyTorch run in that process."""
import subprocess
import sys

import pytest

import cdriver

pytestmark = [pytest.mark.gpu]


@pytest.mark.parametrize("seed", [1, 2])
def test_c_program_matches_oracle(seed):
    exe = cdriver.build()
    print(f"c_abi_step seed {seed}, 12 steps", file=sys.stderr, flush=True)
    r = subprocess.run([exe, str(seed), "12"], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, file=sys.stderr, flush=True)
    if r.returncode == 77:
        pytest.skip("no GPU")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all bars met" in r.stdout

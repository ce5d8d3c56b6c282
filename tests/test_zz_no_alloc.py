"""rikfad_friction_report_noalloc against rikfad_friction_report.

The no-allocation variant runs the report's kernels on the library's
static device workspace instead of a per-call allocation.  Two calls in a
row, the second on a smaller tensor (so the workspace still holds the
first call's values), must each give the existing entry point's results
bit for bit, and the oracle's to the diagnostic's tolerance.  The friction
tensors are drawn on the host (never by the GPU path)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_30342_amd import rikfad as R

from parity import log

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

KEYS = ("xi_fro2", "err_fro2", "sum_r", "sigma1", "rel_err", "eckart_young_floor", "stable_rank",
        "power_iters")


def _mixture(m, n, k, seed):
    rng = np.random.default_rng(seed)
    xi = sum(np.outer(rng.random(m), rng.random(n)) for _ in range(k))
    return (xi + 0.05 * rng.random((m, n))).astype(np.float32)


# The GPT2-S embedding's shape first, then a smaller tensor whose one-pass
# and two-pass regions of the workspace overlap the first call's.
SHAPES = [(50257, 768, 3, 21), (300, 1025, 2, 22)]


def test_noalloc_report_equals_allocating_report_twice():
    s = torch.cuda.current_stream().cuda_stream
    limit = R.rikfad_friction_report_noalloc_max_bytes()
    for m, n, k, seed in SHAPES:
        need = R.rikfad_friction_report_workspace_bytes(m, n)
        log(f"[case] friction report noalloc {m}x{n} workspace={need} of {limit} bytes")
        assert 0 < need <= limit
        xi = _mixture(m, n, k, seed)
        d = torch.from_numpy(xi).cuda()
        want = R.rikfad_friction_report(d.data_ptr(), m, n, 1e-8, 40, s)
        got = R.rikfad_friction_report_noalloc(d.data_ptr(), m, n, 1e-8, 40, s)
        for key in KEYS:
            assert got[key] == want[key], (key, got[key], want[key])
        ref = O.friction_report(xi.astype(np.float64), 1e-8)
        for key in ("xi_fro2", "sum_r", "sigma1"):
            assert got[key] == pytest.approx(ref[key], rel=1e-9), key
        assert got["rel_err"] == pytest.approx(ref["rel_err"], rel=1e-7, abs=1e-7)
        del d

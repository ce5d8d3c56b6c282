"""GPU parity of the rank-1 friction diagnostic (Section 4) against the fp64
oracle.  The friction tensors come from the oracle's own element-wise iKFAD
trajectories on seeded synthetic gradients (never from the GPU path) and are
rounded to fp32 before both sides see them."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_30342_amd import rikfad as R
from paper_2609_30342_amd import synth

from parity import log

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

KEYS = ("xi_fro2", "err_fro2", "sum_r", "sigma1", "rel_err", "eckart_young_floor", "stable_rank")


def _ikfad_friction(m, n, steps, seed, hp):
    wl = synth.Workload([synth.TensorSpec("w", m, n)], seed=seed)
    x = wl.x0(0).astype(np.float64).ravel()
    p, xi = np.zeros(m * n), np.zeros(m * n)
    for s in range(steps):
        O.ikfad_step(x, wl.grad(0, s).astype(np.float64).ravel(), p, xi, O.HParams(**hp))
    return xi.reshape(m, n).astype(np.float32)


def _mixture(m, n, k, seed):
    rng = np.random.default_rng(seed)
    xi = sum(np.outer(rng.random(m), rng.random(n)) for _ in range(k))
    return (xi + 0.05 * rng.random((m, n))).astype(np.float32)


CASES = [
    ("ikfad_384x1152", lambda: _ikfad_friction(384, 1152, 20, 1, synth.HP_FRICTION), 1e-8),
    ("ikfad_1536x384", lambda: _ikfad_friction(1536, 384, 20, 2, synth.HP_FRICTION), 0.0),
    ("ikfad_ragged", lambda: _ikfad_friction(77, 27, 10, 3, synth.HP_FRICTION), 1e-8),
    ("mixture3_300x520", lambda: _mixture(300, 520, 3, 4), 1e-8),
    ("mixture5_4097x64", lambda: _mixture(4097, 64, 5, 5), 0.0),
    ("single_row", lambda: _mixture(1, 300, 1, 6), 0.0),
    ("mixture2_700x1000", lambda: _mixture(700, 1000, 2, 7), 1e-8),    # widest one-pass rows
    ("mixture2_300x1025", lambda: _mixture(300, 1025, 2, 8), 1e-8),    # two-pass iteration
    # each register width of the one-pass iteration filled exactly, with a
    # ragged last block of rows
    ("mixture2_129x256", lambda: _mixture(129, 256, 2, 9), 1e-8),
    ("mixture2_257x512", lambda: _mixture(257, 512, 2, 10), 0.0),
    ("mixture3_1000x768", lambda: _mixture(1000, 768, 3, 11), 1e-8),
]


@pytest.mark.parametrize("name,make,eps", CASES, ids=[c[0] for c in CASES])
def test_friction_report_matches_oracle(name, make, eps):
    xi = make()
    m, n = xi.shape
    log(f"[case] friction report {name} {m}x{n} eps={eps}")
    want = O.friction_report(xi.astype(np.float64), eps)
    d = torch.from_numpy(xi).cuda()
    got = R.rikfad_friction_report(d.data_ptr(), m, n, eps, 200,
                                   torch.cuda.current_stream().cuda_stream)
    log(f"[diag] {name} gpu={ {k: round(got[k], 6) for k in ('rel_err', 'eckart_young_floor', 'stable_rank')} } "
        f"oracle={ {k: round(want[k], 6) for k in ('rel_err', 'eckart_young_floor', 'stable_rank')} }")
    for k in ("xi_fro2", "sum_r", "sigma1", "stable_rank"):
        assert got[k] == pytest.approx(want[k], rel=1e-9, abs=1e-300), k
    # exactly rank-1 inputs leave only rounding noise in |xi - xi~|^2
    assert got["err_fro2"] == pytest.approx(want["err_fro2"], rel=1e-9, abs=1e-12 * want["xi_fro2"])
    # the floor sqrt(1 - s^2/F) loses digits when it is tiny: absolute bound
    assert got["rel_err"] == pytest.approx(want["rel_err"], rel=1e-7, abs=1e-7)
    assert got["eckart_young_floor"] == pytest.approx(want["eckart_young_floor"], abs=1e-6)
    assert got["rel_err"] >= got["eckart_young_floor"] - 1e-6


def test_friction_report_rejects_bad_arguments():
    d = torch.zeros(8, device="cuda")
    with pytest.raises(R.RikfadError):
        R.rikfad_friction_report(d.data_ptr(), 0, 8)
    with pytest.raises(R.RikfadError):
        R.rikfad_friction_report(d.data_ptr() + 2, 2, 2)
    with pytest.raises(R.RikfadError):
        R.rikfad_friction_report(d.data_ptr(), 2, 4, power_iters=0)

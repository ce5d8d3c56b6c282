"""The benchmarks' kernel timing: start / stop events attached to the first
and last dispatch of each phase of a step.  Counts of timed steps, phases
that do and do not run (no finalisation for a set of vectors, the apply
phase only in two-pass mode), pausing and resuming the record, and that a
read clears it.  Times are checked for sign and order of magnitude only."""
import pytest
import torch

from paper_2609_30342_amd import rikfad as R
from paper_2609_30342_amd import synth

from parity import log

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _tensors(shapes, dtype=torch.float32):
    gen = torch.Generator(device="cuda:0").manual_seed(5)
    xs = [torch.randn(s, generator=gen, device="cuda:0").to(dtype) for s in shapes]
    gs = [torch.randn(s, generator=gen, device="cuda:0").to(dtype) for s in shapes]
    return xs, gs


@pytest.mark.parametrize("two_pass", [False, True])
def test_rikfad_timing_phases_and_pause(two_pass):
    log(f"[case] rikfad timing two_pass={two_pass}")
    xs, gs = _tensors([(256, 512), (1, 512), (4200, 96)])
    opt = R.RIKFAD(xs, gs, two_pass=two_pass, **synth.HP_BASE)
    opt.step()
    k1, k2, k3, n = R.rikfad_timing_read(opt.ctx)          # nothing timed yet
    assert (k1, k2, k3, n) == (0.0, 0.0, 0.0, 0)
    R.rikfad_timing_enable(opt.ctx, True)
    opt.step()
    opt.step()
    R.rikfad_timing_enable(opt.ctx, False)
    opt.step()                                             # not timed
    R.rikfad_timing_enable(opt.ctx, True)                  # the record is kept
    opt.step()
    R.rikfad_timing_enable(opt.ctx, False)
    k1, k2, k3, n = R.rikfad_timing_read(opt.ctx)
    assert n == 3
    assert 0.0 < k1 < 100.0 and 0.0 < k2 < 100.0
    assert (k3 > 0.0) if two_pass else (k3 == 0.0)
    assert R.rikfad_timing_read(opt.ctx) == (0.0, 0.0, 0.0, 0)   # cleared
    opt.close()


def test_rikfad_timing_vectors_only_has_no_finalisation():
    log("[case] rikfad timing vectors only")
    xs, gs = _tensors([(1, 1000), (300, 1)])
    opt = R.RIKFAD(xs, gs, **synth.HP_BASE)
    R.rikfad_timing_enable(opt.ctx, True)
    for _ in range(4):
        opt.step()
    k1, k2, k3, n = R.rikfad_timing_read(opt.ctx)
    assert n == 4 and k1 > 0.0 and k2 == 0.0 and k3 == 0.0
    opt.close()


def test_rikfad_timing_two_storage_types():
    """fp32 and bf16 tensors: two streaming launches, timed as one phase."""
    log("[case] rikfad timing fp32 + bf16")
    x32, g32 = _tensors([(512, 512)])
    x16, g16 = _tensors([(512, 512)], torch.bfloat16)
    opt = R.RIKFAD(x32 + x16, g32 + g16, **synth.HP_BASE)
    R.rikfad_timing_enable(opt.ctx, True)
    opt.step()
    opt.step()
    k1, k2, k3, n = R.rikfad_timing_read(opt.ctx)
    assert n == 2 and k1 > 0.0 and k2 > 0.0 and k3 == 0.0
    opt.close()


def test_ikfad_and_adafm_timing():
    log("[case] ikfad / adafm timing")
    xs, gs = _tensors([(256, 512), (1, 512)])
    ik = R.IKFAD(xs, gs, h=1e-3)
    R.ikfad_timing_enable(ik.ctx, True)
    ik.step()
    ik.step()
    ms, n = R.ikfad_timing_read(ik.ctx)
    assert n == 2 and 0.0 < ms < 100.0
    ik.close()
    for clip in (1.0, 0.0):
        opt = R.ADAFM(xs, gs, h=1e-3, clip_threshold=clip)
        R.adafm_timing_enable(opt.ctx, True)
        for _ in range(3):
            opt.step()
        ms5, n = R.adafm_timing_read(opt.ctx)
        assert n == 3, n
        stats, fin, rms, scale, upd = ms5
        assert stats > 0.0 and fin > 0.0 and scale > 0.0 and upd > 0.0, ms5
        assert (rms > 0.0) == (clip > 0.0), ms5       # no RMS pass without clipping
        opt.close()

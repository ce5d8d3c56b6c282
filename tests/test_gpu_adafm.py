"""GPU parity of the Adafactor-m step (the paper's baseline optimiser,
Section 2, Methodology, left-hand system; schedule beta2_t = 1 - t^{-0.8},
Section 3 and App. "Hyperparameters") through the C ABI against the fp64
oracle, on the same seeded synthetic workloads as the R-iKFAD tests.

Tolerances are those of the R-iKFAD parity tests: x and the first moment M
normwise and element-wise (with the rms floor) 1e-5, the factors R, C and
the unfactored second moment of vectors plain relative 1e-5, bf16 x against
the oracle's unrounded update 4e-3.  Every case prints its name first.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_30342_amd import rikfad as R
from paper_2609_30342_amd import synth

from parity import (adafm_oracle_step, assert_ok, compare_adafm, log, make_adafm_pair,
                    run_adafm_parity)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

S = synth.TensorSpec
HP = dict(h=1e-3, beta1=0.9)          # decay -0.8, eps1 1e-30, clipping at 1, no scaling


def test_single_matrix():
    log("[case] adafm single 256x512")
    _, errs = run_adafm_parity(synth.single_matrix(), HP, 8, label="single")
    assert_ok(errs, label="adafm single")


MIXED = [S("a", 96, 200), S("b", 1, 200), S("c", 40, 640, "bf16"), S("d", 640, 1, "bf16"),
         S("e", 300, 27)]


@pytest.mark.parametrize("variant", ["clip_active", "scaled", "scaled_no_clip", "beta1_zero"])
def test_options(variant):
    """Update clipping that bites (d = 0.5), the parameter scale
    max(eps2, RMS(X)) with and without clipping, and beta1 = 0."""
    hp = dict(HP, **{"clip_active": dict(clip_threshold=0.5),
                     "scaled": dict(scale_parameter=True),
                     "scaled_no_clip": dict(scale_parameter=True, clip_threshold=0.0),
                     "beta1_zero": dict(beta1=0.0)}[variant])
    log(f"[case] adafm options {variant} {hp}")
    _, errs = run_adafm_parity(MIXED, hp, 5, seed=2, label=variant)
    assert_ok(errs, label=variant)


def _random_set(seed):
    """2 to 7 tensors of random shape (vectors, narrow and ragged, wide,
    tall), fp32 or bf16, random options, aligned or misaligned."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0xADA])))
    specs = []
    for i in range(int(rng.integers(2, 8))):
        kind = int(rng.integers(0, 4))
        if kind == 0:
            k = int(rng.integers(1, 2000))
            m, n = (1, k) if rng.random() < 0.5 else (k, 1)
        elif kind == 1:
            m, n = int(rng.integers(1, 600)), int(rng.integers(2, 70))
        elif kind == 2:
            m, n = int(rng.integers(1, 80)), int(rng.integers(200, 3000))
        else:
            m, n = int(rng.integers(600, 5000)), int(rng.integers(2, 300))
        specs.append(S(f"t{i}", m, n, "bf16" if rng.random() < 0.4 else "fp32"))
    hp = dict(h=float(rng.choice([1e-3, 1e-2])), beta1=float(rng.choice([0.0, 0.9])),
              clip_threshold=float(rng.choice([0.0, 0.5, 1.0])),
              scale_parameter=bool(rng.random() < 0.5))
    return specs, hp, int(rng.random() < 0.3), int(rng.choice([1, 1, 50]))


@pytest.mark.parametrize("seed", range(8))
def test_random_sets(seed):
    """Seeded random parameter sets against the oracle, 4 steps each, some
    starting late in the beta2 schedule."""
    specs, hp, x_offset, t0 = _random_set(seed)
    log(f"[case] adafm random set seed={seed} x_offset={x_offset} t0={t0} hp={hp} "
        f"{[(s.m, s.n, s.dtype) for s in specs]}")
    _, errs = run_adafm_parity(specs, hp, 4, seed=seed, x_offset=x_offset, first_step=t0,
                               label=f"random {seed}")
    assert_ok(errs, label=f"adafm random {seed}")


EDGE = [
    ("ragged_n27", [S("a", 300, 27)]),
    ("wide_ragged", [S("a", 257, 1000)]),
    ("narrow_L16", [S("a", 513, 64)]),
    ("narrow_L2", [S("a", 70, 8)]),
    ("tiny", [S("a", 5, 6), S("b", 2, 2), S("c", 2, 3)]),
    ("vectors", [S("v", 1, 1000), S("w", 1000, 1), S("s", 1, 1), S("u", 1, 7)]),
    ("bf16_v4", [S("a", 64, 36, "bf16"), S("b", 200, 776, "bf16")]),
    ("bf16_v1", [S("a", 65, 27, "bf16"), S("b", 1, 33, "bf16")]),
    ("tall", [S("a", 3000, 12), S("b", 2100, 100)]),
    ("very_wide", [S("a", 40, 50257), S("b", 1, 50257)]),
    ("many_small", [S(f"t{i}", 3 + i % 5, 5 + i % 7) for i in range(300)]
                   + [S(f"v{i}", 1, 1 + i % 9) for i in range(300)]),
]


@pytest.mark.parametrize("name,specs", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes(name, specs):
    log(f"[case] adafm edge {name} {[(s.m, s.n, s.dtype) for s in specs]}")
    _, errs = run_adafm_parity(specs, HP, 6, seed=3, label=f"edge {name}")
    assert_ok(errs, label=name)


# bf16 matrices whose rows allow 8-byte accesses take 4 elements per lane
# in all three passes, the others the one-column path, in the same launch
# with the set's vectors; with x_offset = 2 elements (4 bytes) every bf16
# row loses the 8-byte alignment and every matrix takes the one-column path.
BF16_WIDTHS = [S("w4a", 200, 776, "bf16"), S("w4", 64, 36, "bf16"), S("w1", 65, 27, "bf16"),
               S("v", 1, 333, "bf16"), S("w4b", 33, 1024, "bf16"), S("f", 70, 96)]


@pytest.mark.parametrize("x_offset", [0, 2])
def test_bf16_read_widths(x_offset):
    log(f"[case] adafm bf16 read widths x_offset={x_offset} "
        f"{[(s.m, s.n, s.dtype) for s in BF16_WIDTHS]}")
    _, errs = run_adafm_parity(BF16_WIDTHS, dict(HP, clip_threshold=0.5), 6, seed=6,
                               x_offset=x_offset, label=f"bf16 widths off={x_offset}")
    assert_ok(errs, label="bf16 read widths")


def test_misaligned_views_take_scalar_path():
    specs = [S("a", 33, 64), S("b", 1, 50), S("c", 20, 20, "bf16")]
    log("[case] adafm misaligned views")
    _, errs = run_adafm_parity(specs, HP, 4, seed=4, x_offset=1, label="misaligned")
    assert_ok(errs, label="misaligned")


def test_late_schedule_after_set_step():
    """Resuming at t = 1000 (beta2_t close to 1) through adafm_set_step."""
    log("[case] adafm t = 1000..1002")
    pair, errs = run_adafm_parity(MIXED, HP, 3, seed=6, first_step=1000, label="late")
    assert_ok(errs, label="late schedule")
    assert R.adafm_get_step(pair.opt.ctx) == 1002


def test_gpt2_nano():
    log("[case] adafm gpt2_nano fp32")
    _, errs = run_adafm_parity(synth.gpt2_nano(), HP, 5, label="gpt2_nano")
    assert_ok(errs, label="gpt2_nano")


def test_tinyvit_bf16():
    log("[case] adafm tinyvit bf16")
    _, errs = run_adafm_parity(synth.tinyvit_like(), HP, 4, label="tinyvit")
    assert_ok(errs, label="tinyvit")


def test_many_tiny_tensors():
    """2,000 tensors of 1 to 40 rows and columns, fp32 and bf16, with
    clipping and parameter scaling on: per-tensor RMS and scale over
    thousands of small tiles, against the oracle."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([13, 0xADA])))
    specs = [S(f"t{i}", int(rng.integers(1, 41)), int(rng.integers(1, 41)),
               "bf16" if rng.random() < 0.4 else "fp32") for i in range(2000)]
    log(f"[case] adafm many tiny tensors: {len(specs)}")
    hp = dict(HP, clip_threshold=0.5, scale_parameter=True)
    _, errs = run_adafm_parity(specs, hp, 4, seed=13, label="many tiny")
    assert_ok(errs, label="adafm many tiny")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_gpt2_small_full_size(dtype):
    """GPT2-S-shaped set at full size in one context (the benchmark's
    configuration); the oracle follows the embeddings, block 0 and some
    vectors; 3 steps."""
    specs = synth.gpt2_small(dtype)
    names = {"wte", "wpe", "h0.attn.qkv", "h0.mlp.proj", "h0.ln_1.w", "h11.mlp.fc.b"}
    checked = [i for i, s in enumerate(specs) if s.name in names]
    log(f"[case] adafm gpt2_small {dtype} checked={len(checked)}")
    _, errs = run_adafm_parity(specs, HP, 3, checked=checked, label=f"gpt2_small {dtype}")
    assert_ok(errs, label="adafm gpt2_small")


def test_zero_gradient_rows_and_columns_with_eps1_zero():
    """eps1 = 0 and a gradient with zero rows and columns: the estimate is 0
    there and U is taken as 0 (no 0/0), on both sides."""
    specs = [S("a", 40, 72), S("v", 1, 64)]
    hp = dict(HP, eps1=0.0)
    log("[case] adafm zero rows/cols eps1=0")
    pair = make_adafm_pair(specs, hp, seed=7)
    rng = np.random.default_rng(7)
    for t in range(1, 4):
        hg = {}
        for i, sp in enumerate(specs):
            g = rng.standard_normal((sp.m, sp.n)).astype(np.float32).astype(np.float64)
            if sp.m > 1:
                g[3, :] = 0.0
                g[:, 10] = 0.0
            else:
                g[0, :5] = 0.0
            hg[i] = g
            pair.gs[i].copy_(torch.from_numpy(g).to(torch.float32))
        pair.opt.step()
        adafm_oracle_step(pair, hg, t, hp)
        errs = compare_adafm(pair)
        assert_ok(errs, label=f"zero rows t={t}")
    for x in pair.xs:
        assert torch.isfinite(x).all()


def _run(specs, hp, steps, seed):
    pair = make_adafm_pair(specs, hp, seed=seed, checked=[])
    rng = np.random.default_rng(seed)
    for _ in range(steps):
        for g in pair.gs:
            g.copy_(torch.from_numpy(rng.standard_normal(tuple(g.shape))).to(g.dtype))
        pair.opt.step()
    torch.cuda.synchronize()
    return pair


def test_deterministic_bitwise():
    log("[case] adafm determinism")
    a = _run(MIXED, HP, 4, 11)
    b = _run(MIXED, HP, 4, 11)
    for i in range(len(MIXED)):
        assert torch.equal(a.xs[i], b.xs[i])
        for u, v in zip(a.opt.state[i], b.opt.state[i]):
            assert torch.equal(u, v)


def test_checkpoint_resume_bitwise():
    """6 steps == 3 steps, save (x, M, R, C, step count), new context, 3 more."""
    log("[case] adafm checkpoint/resume")
    specs = MIXED
    full = _run(specs, HP, 6, 12)
    rng = np.random.default_rng(12)
    first = make_adafm_pair(specs, HP, seed=12, checked=[])
    for _ in range(3):
        for g in first.gs:
            g.copy_(torch.from_numpy(rng.standard_normal(tuple(g.shape))).to(g.dtype))
        first.opt.step()
    torch.cuda.synchronize()
    saved_x = [x.clone() for x in first.xs]
    saved = [tuple(t.clone() for t in st) for st in first.opt.state]
    steps = first.opt.steps_taken
    first.opt.close()
    gs = [torch.empty_like(x) for x in saved_x]
    opt = R.ADAFM(saved_x, gs, state=saved, **HP)
    R.adafm_set_step(opt.ctx, steps)
    for _ in range(3):
        for g in gs:
            g.copy_(torch.from_numpy(rng.standard_normal(tuple(g.shape))).to(g.dtype))
        opt.step()
    torch.cuda.synchronize()
    for i in range(len(specs)):
        assert torch.equal(full.xs[i], saved_x[i])
        for u, v in zip(full.opt.state[i], saved[i]):
            assert torch.equal(u, v)


def test_nonfinite_gradient_is_flagged():
    log("[case] adafm non-finite flag")
    specs = [S("a", 16, 32)]
    pair = make_adafm_pair(specs, HP, seed=13, checked=[])
    pair.gs[0].normal_()
    pair.opt.step()
    assert not R.adafm_nonfinite(pair.opt.ctx)
    pair.gs[0][2, 3] = float("inf")
    pair.opt.step()
    assert R.adafm_nonfinite(pair.opt.ctx)


def test_byte_counts():
    """The update pass moves 20 B per fp32 matrix element and R, C once;
    the whole step adds two gradient reads (statistics and RMS) and the
    factor update."""
    specs = [S("a", 64, 128), S("b", 1, 100), S("c", 32, 48, "bf16")]
    log("[case] adafm byte counts")
    pair = make_adafm_pair(specs, HP, checked=[])
    total, upd, state = R.adafm_min_bytes(pair.opt.ctx)
    assert upd == 64 * 128 * 20 + 4 * (64 + 128) + 100 * 24 + 32 * 48 * 14 + 4 * (32 + 48)
    assert total == (64 * 128 * 28 + 8 * (64 + 128) + 100 * 36
                     + 32 * 48 * 18 + 8 * (32 + 48))
    assert state == 4 * 64 * 128 + 4 * (64 + 128) + 8 * 100 + 4 * 32 * 48 + 4 * (32 + 48)

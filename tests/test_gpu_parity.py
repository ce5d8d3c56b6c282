"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Every case prints its name, shapes and seed before touching the GPU.
Workloads are the seeded synthetic parameter sets of
paper_2609_30342_amd.synth (shapes of the paper's four models, Section 4).
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_30342_amd import rikfad as R
from paper_2609_30342_amd import synth

from parity import (TOL_F32, assert_ok, compare, host, load_grads, log, make_pair,
                    oracle_step, rel_plain, rel_rms, run_parity)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

S = synth.TensorSpec


def test_library_is_the_native_hip_build():
    """The library these tests call is the in-tree build, mapped into this
    process, carrying gfx950 code, and its kernels run on the GPU (a probe
    copies device memory)."""
    import os
    R.lib()
    path = os.path.realpath(R.LIB_PATH)
    assert os.path.dirname(path) == os.path.realpath(
        os.path.join(os.path.dirname(__file__), "..", "paper_2609_30342_amd"))
    with open("/proc/self/maps") as f:
        assert path in f.read()
    with open(path, "rb") as f:
        assert b"gfx950" in f.read()
    n = 1 << 16
    a = torch.arange(n, device="cuda", dtype=torch.float32)
    b = torch.zeros_like(a)
    R.rikfad_probe_copy(a.data_ptr(), b.data_ptr(), 4 * n,
                        torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# ------------------------------------------------------------- config 0

@pytest.mark.parametrize("two_pass", [False, True])
def test_single_matrix_base(two_pass):
    """256 x 512 fp32, h = 1e-3, gamma = 0, alpha = 0.1, mu = 1, eps = 1e-8, 20 steps."""
    log(f"[case] single 256x512 base two_pass={two_pass}")
    _, errs = run_parity(synth.single_matrix(), synth.HP_BASE, 20, two_pass=two_pass,
                         label=f"single base two_pass={two_pass}")
    assert_ok(errs, label="single base")


@pytest.mark.parametrize("gamma", [0.0, 0.05])
def test_single_matrix_friction_active(gamma):
    """Same matrix with friction strong enough that the half-kicks matter
    (median (h/2) xi~ around 0.1 by the end), with and without damping D."""
    hp = dict(synth.HP_FRICTION, gamma=gamma)
    log(f"[case] single 256x512 friction gamma={gamma}")
    pair, errs = run_parity(synth.single_matrix(), hp, 50, label=f"single friction g={gamma}")
    assert_ok(errs, label="single friction")
    o = pair.ref[0]
    xi = O.rank1_friction(o.r, o.c, hp["eps_stab"])
    assert np.median(0.5 * hp["h"] * xi) > 0.02      # the friction path is exercised


# The host folds the hyperparameters into e^{-alpha h}, (1 - e^{-alpha h}) /
# (mu alpha), e^{-gamma h} and h once per set_hparams (Section 2, the factor
# filter's exact solution).  Limits of that computation, each with kappa
# near 1 so the friction stays active:
COEFF_CASES = [
    # alpha = 0: the factors integrate (P^(1))^2 without decay, kappa = h / mu
    ("alpha_0", dict(h=0.1, gamma=0.0, alpha=0.0, mu=0.1, eps_stab=1e-8)),
    # alpha h = 1e-7: 1 - e^{-alpha h} survives only through expm1, and
    # e^{-alpha h} is within two fp32 ulps of 1
    ("alpha_h_1e-7", dict(h=0.1, gamma=0.0, alpha=1e-6, mu=0.1, eps_stab=1e-8)),
    # strong damping: e^{-gamma h} = e^{-1/2}
    ("gamma_h_0.5", dict(h=0.1, gamma=5.0, alpha=0.1, mu=0.1, eps_stab=1e-8)),
]


@pytest.mark.parametrize("name,hp", COEFF_CASES, ids=[c[0] for c in COEFF_CASES])
def test_coefficient_limits(name, hp):
    specs = [S("a", 300, 520), S("b", 1, 520), S("c", 77, 1000, "bf16"), S("d", 129, 27)]
    log(f"[case] coefficients {name} hp={hp}")
    pair, errs = run_parity(specs, hp, 12, seed=11, label=f"coefficients {name}")
    assert_ok(errs, label=name)
    o = pair.ref[0]
    xi = O.rank1_friction(o.r, o.c, hp["eps_stab"])
    assert np.median(0.5 * hp["h"] * xi) > 0.005     # the friction path is exercised


# ------------------------------------------------------- shapes and tails

EDGE = [
    ("ragged_n27", [S("a", 300, 27)]),                       # n % 4 != 0 -> scalar path
    ("wide_ragged", [S("a", 257, 1000)]),                    # 3 full column blocks + 58 lanes
    ("narrow_L16", [S("a", 513, 64)]),                       # 4 rows per load
    ("narrow_L2", [S("a", 70, 8)]),
    ("narrow_L1", [S("a", 3, 4)]),
    ("tiny", [S("a", 5, 6), S("b", 2, 2), S("c", 2, 3)]),
    ("vectors", [S("v", 1, 1000), S("w", 1000, 1), S("s", 1, 1), S("u", 1, 7)]),
    ("bf16_776", [S("a", 200, 776, "bf16")]),                # 194 lanes: 3 blocks + 2 (L = 2)
    ("bf16_v4", [S("a", 64, 36, "bf16")]),
    ("bf16_v1", [S("a", 65, 27, "bf16"), S("b", 1, 33, "bf16")]),
    ("tall", [S("a", 3000, 12)]),                            # many stripes, 3 lanes per row
    ("mixed", [S("a", 96, 200), S("b", 1, 200), S("c", 40, 640, "bf16"), S("d", 640, 1, "bf16")]),
    ("very_wide", [S("a", 40, 50257), S("b", 1, 50257)]),    # 197 column blocks per row
    ("many_small", [S(f"t{i}", 3 + i % 5, 5 + i % 7) for i in range(300)]
                   + [S(f"v{i}", 1, 1 + i % 9) for i in range(300)]),
]


@pytest.mark.parametrize("name,specs", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes(name, specs):
    log(f"[case] edge {name} {[(s.m, s.n, s.dtype) for s in specs]}")
    _, errs = run_parity(specs, synth.HP_FRICTION, 12, seed=3, label=f"edge {name}")
    assert_ok(errs, label=name)


def _random_set(seed):
    """2 to 7 tensors of random shape (vectors, narrow and ragged, wide,
    tall), fp32 or bf16, random hyperparameters, aligned or misaligned."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x5E7])))
    specs = []
    for i in range(int(rng.integers(2, 8))):
        kind = int(rng.integers(0, 4))
        if kind == 0:                                    # vector, either orientation
            k = int(rng.integers(1, 2000))
            m, n = (1, k) if rng.random() < 0.5 else (k, 1)
        elif kind == 1:                                  # narrow, often not 4-aligned
            m, n = int(rng.integers(1, 600)), int(rng.integers(2, 70))
        elif kind == 2:                                  # wide, ragged last block
            m, n = int(rng.integers(1, 80)), int(rng.integers(200, 3000))
        else:                                            # tall: many row stripes
            m, n = int(rng.integers(600, 5000)), int(rng.integers(2, 300))
        specs.append(S(f"t{i}", m, n, "bf16" if rng.random() < 0.4 else "fp32"))
    hp = dict(h=float(rng.choice([1e-3, 0.05, 0.1])), gamma=float(rng.choice([0.0, 0.05])),
              alpha=float(rng.choice([0.0, 0.1, 0.5])), mu=float(rng.choice([0.1, 1.0])),
              eps_stab=float(rng.choice([0.0, 1e-8, 0.1])))
    return specs, hp, int(rng.random() < 0.3)


@pytest.mark.parametrize("seed", range(16))
def test_random_sets(seed):
    """Seeded random parameter sets against the oracle, 6 steps each."""
    specs, hp, x_offset = _random_set(seed)
    log(f"[case] random set seed={seed} x_offset={x_offset} hp={hp} "
        f"{[(s.m, s.n, s.dtype) for s in specs]}")
    _, errs = run_parity(specs, hp, 6, seed=seed, x_offset=x_offset, label=f"random {seed}")
    assert_ok(errs, label=f"random {seed}")


def test_many_tiny_tensors():
    """3,000 tensors of 1 to 40 rows and columns (vectors, one-column and
    4-wide matrices, fp32 and bf16) in one context: one launch per storage
    type over thousands of small tiles, against the oracle."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([11, 0x7E1])))
    specs = [S(f"t{i}", int(rng.integers(1, 41)), int(rng.integers(1, 41)),
               "bf16" if rng.random() < 0.4 else "fp32") for i in range(3000)]
    log(f"[case] many tiny tensors: {len(specs)}, {sum(sp.numel for sp in specs)} elements")
    _, errs = run_parity(specs, synth.HP_FRICTION, 4, seed=11, label="many tiny")
    assert_ok(errs, label="many tiny")


# Column items split their T threads (256, or 1024 when a matrix has more
# than 512 row stripes) into S stripe lanes of T / S threads with 4 columns
# each, S the smallest power of two leaving each thread at most 8 row
# stripes (at least one 16-column group per item); up to 16 stripe lanes
# fold inside a wave, more through LDS.  These sets are small (fewer tiles
# than compute units: 16-row stripes) except "mixed" and the last two:
# S = 8 at 64 stripes (1024 rows), S = 16 at 66 (1056 rows, and "mixed"),
# S = 32 at 132-141, S = 64 at 300 (the cap of 256-thread items: one
# 16-column group each), S = 128 at 625 (20000 rows), and S = 256 with two
# batches of loads per thread at 2188 stripes (70000 rows).  The edge
# shapes above cover S = 1, 2 and 4.
COLUMN_CASES = [
    ("s8_64_stripes", [S("a", 1024, 300)], 12),
    ("s16_66_stripes", [S("a", 1056, 300)], 12),
    ("tall_s32", [S("a", 9000, 64), S("b", 4200, 96, "bf16")], 12),
    ("mixed", [S("a", 96, 200), S("b", 1, 200), S("c", 40, 640, "bf16"), S("d", 640, 1, "bf16"),
               S("e", 2100, 1000)], 12),
    ("s64_cap_256_threads", [S("a", 9600, 256)], 6),
    ("s256_two_batches", [S("a", 70000, 256), S("b", 1, 256)], 5),
    # 625 stripes: 1024-thread items of 128 stripe lanes x 32 columns, the
    # last of 8 columns; the one-column-path matrix shares the launch size
    ("ragged_1024_threads", [S("a", 20000, 1000), S("b", 300, 27)], 4),
]


@pytest.mark.parametrize("name,specs,steps", COLUMN_CASES, ids=[c[0] for c in COLUMN_CASES])
def test_column_finalisation(name, specs, steps):
    """Tensors from a few to thousands of row stripes, across the column
    items' stripe-lane counts, against the oracle in the friction-active
    setting."""
    log(f"[case] column finalisation {name}")
    _, errs = run_parity(specs, synth.HP_FRICTION, steps, seed=8, label=f"columns {name}")
    assert_ok(errs, label=name)


@pytest.mark.parametrize("m,tiles", [(992, 496), (1024, 256)])
def test_small_set_rows_per_wave_threshold(m, tiles):
    """m x 2048 fp32 just below (992 rows: 248 tiles at 4 rows per wave,
    so the planner takes 2 rows per wave and 496 tiles) and at (1024 rows:
    256 tiles, 4 rows per wave) the fewer-tiles-than-compute-units rule,
    against the oracle in the friction-active setting, 12 steps."""
    log(f"[case] rows-per-wave threshold {m}x2048")
    pair, errs = run_parity([S("a", m, 2048)], synth.HP_FRICTION, 12, seed=6,
                            label=f"threshold {m}x2048")
    assert pair.opt.query()["stream_tiles"] == tiles
    assert_ok(errs, label=f"threshold {m}")


def test_misaligned_views_take_scalar_path():
    """Parameters and gradients that start one element into their buffers
    (not 16-byte aligned) still match the oracle."""
    specs = [S("a", 64, 128), S("b", 1, 64), S("c", 33, 96, "bf16")]
    log("[case] misaligned views")
    pair, errs = run_parity(specs, synth.HP_FRICTION, 8, seed=4, x_offset=1, label="misaligned")
    assert_ok(errs, label="misaligned")


def test_empty_parameter_list_is_a_noop():
    hp = R.hparams(1e-3)
    ctx = R.rikfad_create([], hp)
    R.rikfad_step(ctx)
    R.rikfad_sync_momentum(ctx)
    info = R.rikfad_query(ctx)
    assert info["tensors"] == 0 and info["stream_tiles"] == 0
    R.rikfad_destroy(ctx)


def test_tensor_beyond_2_31_elements():
    """One 50000 x 50000 bf16 tensor (2.5e9 elements: element offsets past
    2^31) with the rank-1 power-of-two gradient g_ij = a_i b_j (exact in
    bf16), x = p = r = c = 0, two steps with the same gradient.  The Table's
    step has closed forms here.  Step 1: xi~ = 0, P^(1) = -h g, X = -h^2 g,
    R_i = kappa h^2 a_i^2 sum_j b_j^2, C_j = kappa h^2 b_j^2 sum_i a_i^2.
    Step 2: E_ij = exp(-(h/2) R_i C_j / (1^T R + eps)), P^(B) = P^(1) E - h g,
    X += h P^(B), P^(1) = P^(B) E, and the factors from its row and column
    sums.  Checked on sampled elements (half in rows past 2^31 / n) and on
    sampled rows of R and columns of C."""
    m = n = 50000
    h, alpha, mu, eps = 0.05, 0.1, 1e-4, 1e-8
    log(f"[case] {m}x{n} bf16 tensor ({m * n} elements)")
    kappa = -np.expm1(-alpha * h) / (mu * alpha)
    arel = np.exp(-alpha * h)
    ia, jb = np.arange(m), np.arange(n)
    a = 2.0 ** (ia % 3 - 1)
    b = 2.0 ** (jb % 5 - 2)
    dev = "cuda:0"
    x = torch.zeros((m, n), dtype=torch.bfloat16, device=dev)
    g = (torch.from_numpy(a.astype(np.float32)).to(dev)[:, None]
         * torch.from_numpy(b.astype(np.float32)).to(dev)[None, :]).to(torch.bfloat16)
    opt = R.RIKFAD([x], [g], h=h, gamma=0.0, alpha=alpha, mu=mu, eps_stab=eps)
    p, r, c = opt.state[0]
    rng = np.random.default_rng(31)
    rows = np.concatenate([rng.integers(0, m, 24), rng.integers(43000, m, 24)])
    cols = rng.integers(0, n, 48)
    ri, cj = torch.from_numpy(rows).to(dev), torch.from_numpy(cols).to(dev)

    def sample(t):
        return t[ri][:, cj].to(torch.float64).cpu().numpy()

    errs = {}

    def check(name, got, want, floor, tol):
        e = float(np.max(np.abs(got - want) / np.maximum(np.abs(want), floor)))
        errs[name] = e
        assert e <= tol, (name, e, errs)

    G = a[rows][:, None] * b[cols][None, :]
    # step 1
    opt.step()
    torch.cuda.synchronize()
    x1 = sample(x)
    P1 = -h * G
    check("x1", x1, -h * h * G, np.sqrt(np.mean((h * h * G) ** 2)), 4e-3)
    check("p1", sample(p), P1, np.sqrt(np.mean(P1 ** 2)), 1e-5)
    R1 = kappa * h * h * a ** 2 * np.sum(b ** 2)
    C1 = kappa * h * h * b ** 2 * np.sum(a ** 2)
    check("r1", r[ri].double().cpu().numpy(), R1[rows], 0.0, 1e-5)
    check("c1", c[cj].double().cpu().numpy(), C1[cols], 0.0, 1e-5)
    # step 2 (same gradient): closed forms from the step-1 factors
    opt.step()
    torch.cuda.synchronize()
    S1 = np.sum(R1)

    def E(i, j):
        return np.exp(-0.5 * h * np.outer(R1[i], C1[j]) / (S1 + eps))

    Es = E(rows, cols)
    PB = P1 * Es - h * G
    check("x2", sample(x), x1 + h * PB, np.sqrt(np.mean((h * PB) ** 2)), 4e-3)
    P2 = PB * Es
    check("p2", sample(p), P2, np.sqrt(np.mean(P2 ** 2)), 1e-5)
    # factors: full row sums for the sampled rows, column sums for the sampled columns
    Er = E(rows, jb)
    rowsq = np.sum((h * a[rows][:, None] * b[None, :] * (Er + 1.0) * Er) ** 2, axis=1)
    Ec = E(ia, cols)
    colsq = np.sum((h * a[:, None] * b[cols][None, :] * (Ec + 1.0) * Ec) ** 2, axis=0)
    check("r2", r[ri].double().cpu().numpy(), arel * R1[rows] + kappa * rowsq, 0.0, 1e-5)
    check("c2", c[cj].double().cpu().numpy(), arel * C1[cols] + kappa * colsq, 0.0, 1e-5)
    log(f"[parity] 50000x50000 errs={ {k: f'{v:.2e}' for k, v in errs.items()} }")
    opt.close()
    del x, g, p, r, c
    torch.cuda.empty_cache()


# ------------------------------------------------------ model-shaped sets

@pytest.mark.parametrize("variant", ["base", "gamma", "eps0"])
def test_gpt2_nano_fp32(variant):
    """GPT2-Nano-shaped parameter set, fp32, 50 steps (base; gamma = 0.1;
    eps_stab = 0, whose first step takes the xi~ = 0 convention)."""
    hp = dict(synth.HP_BASE)
    if variant == "gamma":
        hp["gamma"] = 0.1
    if variant == "eps0":
        hp["eps_stab"] = 0.0
    log(f"[case] gpt2_nano {variant} hp={hp}")
    _, errs = run_parity(synth.gpt2_nano(), hp, 50, label=f"gpt2_nano {variant}")
    assert_ok(errs, label="gpt2_nano")


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_gpt2_nano_fp32_seeds(seed):
    """The 50-step base run on three more seeds: the margin of the
    element-wise bound is known across draws, not from one."""
    log(f"[case] gpt2_nano base seed={seed}")
    _, errs = run_parity(synth.gpt2_nano(), synth.HP_BASE, 50, seed=seed,
                         label=f"gpt2_nano base seed={seed}")
    assert_ok(errs, label=f"gpt2_nano seed {seed}")


def test_gpt2_nano_friction_active():
    log("[case] gpt2_nano friction-active")
    _, errs = run_parity(synth.gpt2_nano(), synth.HP_FRICTION, 30, label="gpt2_nano friction")
    assert_ok(errs, label="gpt2_nano friction")


def test_tinyvit_bf16():
    """Many small tensors (about 150 matrices and their biases, conv kernels
    with n = 27, 576, 1152, 1440), bf16 parameters and gradients, fp32 state."""
    specs = synth.tinyvit_like()
    log(f"[case] tinyvit bf16 tensors={len(specs)}")
    _, errs = run_parity(specs, synth.HP_FRICTION, 20, label="tinyvit bf16")
    assert_ok(errs, label="tinyvit")


def _bf16_order_key(bits):
    """bf16 bit patterns (int16) to integers ordered like their values, so
    that the difference of two keys counts the bf16 values between them."""
    u = bits.astype(np.int64) & 0xFFFF
    return np.where(u & 0x8000, 0x8000 - (u & 0x7FFF), 0x8000 + u)


def test_bf16_independent_trajectories():
    """bf16 parameters stepped on their own, never reset to the oracle's:
    after 20 friction-active steps at least 99.9% of the stored values equal
    the oracle's bit for bit (measured: 99.989%).  A difference starts only
    where the fp32 and the fp64 update fall on the two sides of a rounding
    midpoint, one bf16 spacing (2^-7 relative) at the value's magnitude;
    since the gradients do not depend on x, it keeps its absolute size
    afterwards (several bf16 values apart once the parameter has moved
    towards zero), and a second such event on the same element can add
    another.  The bound checked is two spacings, relative to the value's
    magnitude floored at the tensor's rms (measured: 2 spacings at most)."""
    specs = [S("a", 300, 776, "bf16"), S("b", 64, 1000, "bf16"), S("c", 1, 520, "bf16"),
             S("d", 97, 36, "bf16")]
    log("[case] bf16 independent trajectories, 20 steps")
    hp = synth.HP_FRICTION
    pair = make_pair(specs, hp)
    for s in range(20):
        hg = load_grads(pair, s)
        pair.opt.step()
        oracle_step(pair, hg, hp)
    torch.cuda.synchronize()
    total = equal = 0
    worst = 0
    rel = 0.0
    for i, o in pair.ref.items():
        got = pair.xs[i].view(torch.int16).cpu().numpy().ravel()
        want = torch.from_numpy(o.x.ravel()).to(torch.bfloat16).view(torch.int16).numpy()
        dist = np.abs(_bf16_order_key(got) - _bf16_order_key(want))
        total += dist.size
        equal += int(np.count_nonzero(dist == 0))
        worst = max(worst, int(dist.max()))
        rel = max(rel, rel_rms(host(pair.xs[i]), o.x))
    frac = equal / total
    log(f"[bf16-trajectory] {equal}/{total} bit-equal ({frac:.5%}), "
        f"max {worst} bf16 values apart, rms-floored relative difference {rel:.2e}")
    assert frac >= 0.999, frac
    assert rel <= 2.0 ** -6, rel


def _gpt2s_checked(specs):
    names = {"wte", "wpe", "h0.attn.qkv", "h0.attn.proj", "h0.mlp.fc", "h0.mlp.proj",
             "h0.ln_1.w", "h0.attn.qkv.b", "h11.mlp.fc.b", "ln_f.b"}
    return [i for i, s in enumerate(specs) if s.name in names]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_gpt2_small_full_size(dtype):
    """GPT2-S-shaped set at full size (124.4M parameters, all 148 tensors in
    one launch, the configuration the benchmark times).  The oracle follows
    the embeddings, block 0 and some vectors; 3 steps."""
    specs = synth.gpt2_small(dtype)
    checked = _gpt2s_checked(specs)
    log(f"[case] gpt2_small {dtype} checked={len(checked)}")
    _, errs = run_parity(specs, synth.HP_BASE, 3, checked=checked, label=f"gpt2_small {dtype}")
    assert_ok(errs, label="gpt2_small")


def _assert_friction_active(pair, hp, floor=0.02):
    """Every followed tensor's median (h/2) xi is above `floor`, so rows C.1
    and C.4 of the step act on every element in fp32 (at HP_BASE they round
    to the identity)."""
    for i, o in pair.ref.items():
        xi = o.xi if o.is_vector else O.rank1_friction(o.r, o.c, hp["eps_stab"])
        med = float(np.median(0.5 * hp["h"] * xi))
        assert med > floor, f"{pair.specs[i].name}: median (h/2) xi = {med:.3g}"


@pytest.mark.parametrize("dtype,gamma", [("fp32", 0.0), ("bf16", 0.05)])
def test_gpt2_small_full_size_friction_active(dtype, gamma):
    """The benchmarked GPT2-S set (all 148 tensors in one launch) with the
    friction active: 6 steps at mu = 0.01, and damping D in the bf16 case.
    The oracle follows the embeddings, block 0 and some vectors."""
    specs = synth.gpt2_small(dtype)
    checked = _gpt2s_checked(specs)
    hp = dict(synth.HP_FRICTION_FULL, gamma=gamma)
    log(f"[case] gpt2_small {dtype} friction-active gamma={gamma} checked={len(checked)}")
    pair, errs = run_parity(specs, hp, 6, checked=checked,
                            label=f"gpt2_small {dtype} friction")
    assert_ok(errs, label="gpt2_small friction")
    _assert_friction_active(pair, hp)


def test_distilbert_plus_large_matrices_friction_active():
    """The 1.5B-parameter set (fp32 DistilBERT part, 32 bf16 matrices of
    4096 x 11008 / 11008 x 4096), Student-t(3) row scales, friction active
    (6 steps at mu = 0.01).  The oracle follows the embedding, block 0 and
    two of the large matrices."""
    specs = synth.distilbert_stress()
    names = {"word_emb", "l0.q", "l0.k", "l0.v", "l0.ffn1", "l0.ffn2", "big0", "big1"}
    checked = [i for i, s in enumerate(specs) if s.name in names]
    hp = synth.HP_FRICTION_FULL
    log(f"[case] distilbert+large friction-active checked={len(checked)}")
    pair, errs = run_parity(specs, hp, 6, scales="student_t", checked=checked,
                            label="distilbert stress friction")
    assert_ok(errs, label="distilbert stress friction")
    _assert_friction_active(pair, hp)


def test_distilbert_plus_large_matrices():
    """DistilBERT-shaped fp32 tensors plus 32 bf16 matrices of 4096 x 11008
    and 11008 x 4096 (about 1.5B parameters), Student-t(3) row scales.  The
    oracle follows the DistilBERT part and two of the large matrices."""
    specs = synth.distilbert_stress()
    checked = [i for i, s in enumerate(specs) if not s.name.startswith("big")] + [
        i for i, s in enumerate(specs) if s.name in ("big0", "big1")]
    log(f"[case] distilbert+large tensors={len(specs)} checked={len(checked)}")
    _, errs = run_parity(specs, synth.HP_BASE, 3, scales="student_t", checked=checked,
                         label="distilbert stress")
    assert_ok(errs, label="distilbert stress")


def test_paper_tuned_hyperparameters_saturating_friction():
    """The paper's tuned GPT2-S R-iKFAD0 values (mu = 1.36e-6) with O(1)
    synthetic gradients drive the friction far past exp underflow; the step
    must stay finite and match the oracle."""
    log("[case] tuned hyperparameters")
    specs = [S("a", 384, 1152), S("b", 1, 384)]
    pair, errs = run_parity(specs, synth.HP_GPT2S_TUNED, 10, label="tuned")
    assert_ok(errs, label="tuned")
    assert not pair.opt.nonfinite()


# ------------------------------------------------- special cases (paper)

def test_rank1_momentum_matches_full_ikfad():
    """From P_0 = u v^T with g = 0, R = C = 0 and eps = 0, one R-iKFAD step
    equals one full iKFAD step (the rank-1 friction is exact when [P]^2 is
    rank-1): both HIP paths, compared with each other and with the oracle."""
    m, n = 192, 320
    rng = np.random.default_rng(12)
    u, v = rng.standard_normal(m), rng.standard_normal(n)
    p0 = np.outer(u, v).astype(np.float32)
    hp = dict(h=0.3, gamma=0.2, alpha=0.5, mu=0.25, eps_stab=0.0)
    log("[case] rank-1 identity")
    x = torch.zeros((m, n), device="cuda")
    g = torch.zeros_like(x)
    p = torch.from_numpy(p0).cuda()
    r = torch.zeros(m, device="cuda")
    c = torch.zeros(n, device="cuda")
    opt = R.RIKFAD([x], [g], state=[(p, r, c)], **hp)
    opt.step()
    opt.sync_momentum()
    x2 = torch.zeros_like(x)
    ik = R.IKFAD([x2], [g], h=hp["h"], gamma=hp["gamma"], alpha=hp["alpha"], mu=hp["mu"])
    ik.state[0][0].copy_(torch.from_numpy(p0))
    ik.step()
    torch.cuda.synchronize()
    o = O.make_tensor(np.zeros((m, n)), p0=p0.astype(np.float64))
    O.rikfad_matrix_step(o.x, np.zeros((m, n)), o.p, o.r, o.c, O.HParams(**hp))
    assert rel_rms(host(p), o.p) < TOL_F32
    assert rel_rms(host(ik.state[0][0]), o.p) < TOL_F32
    assert rel_rms(host(p), host(ik.state[0][0])) < TOL_F32
    xi_full = host(ik.state[0][1])
    xi_rank1 = O.rank1_friction(host(r), host(c), 0.0)
    assert rel_rms(xi_rank1, xi_full) < 1e-5


def test_pure_decay_through_library():
    """P = 0, g = 0, eps = 0: the factors only relax and xi~ decays as
    e^{-alpha t} (eqs. rikfad_R, rikfad_C with no forcing)."""
    m, n, steps = 300, 200, 40
    hp = dict(h=0.1, gamma=0.0, alpha=0.6, mu=1.0, eps_stab=0.0)
    rng = np.random.default_rng(13)
    r0 = rng.random(m).astype(np.float32)
    c0 = rng.random(n).astype(np.float32)
    log("[case] pure decay")
    x = torch.zeros((m, n), device="cuda")
    g = torch.zeros_like(x)
    st = (torch.zeros_like(x), torch.from_numpy(r0).cuda(), torch.from_numpy(c0).cuda())
    opt = R.RIKFAD([x], [g], state=[st], **hp)
    for _ in range(steps):
        opt.step()
    opt.sync_momentum()
    torch.cuda.synchronize()
    decay = np.exp(-hp["alpha"] * hp["h"] * steps)
    xi0 = O.rank1_friction(r0.astype(np.float64), c0.astype(np.float64), 0.0)
    xi = O.rank1_friction(host(st[1]), host(st[2]), 0.0)
    assert rel_plain(xi, decay * xi0) < 2e-5
    assert torch.count_nonzero(st[0]) == 0


# ------------------------------------------------------ library behaviour

def _run_steps(specs, hp, steps, two_pass=False, seed=5):
    pair = make_pair(specs, hp, seed=seed, two_pass=two_pass, checked=[])
    for s in range(steps):
        load_grads(pair, s, seed)
        pair.opt.step()
    pair.opt.sync_momentum()
    torch.cuda.synchronize()
    return pair


SPECS_MIX = [S("a", 300, 520), S("b", 1, 520), S("c", 77, 1000, "bf16"), S("d", 129, 27),
             S("e", 4200, 96)]          # e: 66 row stripes, 4 stripe lanes per column item


def test_deterministic_bitwise():
    log("[case] determinism")
    a = _run_steps(SPECS_MIX, synth.HP_FRICTION, 6)
    b = _run_steps(SPECS_MIX, synth.HP_FRICTION, 6)
    for i in range(len(SPECS_MIX)):
        assert torch.equal(a.xs[i], b.xs[i])
        for u, v in zip(a.opt.state[i], b.opt.state[i]):
            assert torch.equal(u, v)


def test_two_contexts_on_two_streams_bitwise():
    """Two contexts stepped at the same time on two streams give, bit for
    bit, what each gives when it runs alone: a context's tables, workspace,
    flag and pending state are its own."""
    specs_b = [S("f", 640, 768), S("g", 1, 768), S("h", 96, 2048, "bf16"), S("k", 33, 27)]
    hp = synth.HP_FRICTION
    log("[case] two contexts on two streams")

    def run(concurrent):
        a = make_pair(SPECS_MIX, hp, seed=5, checked=[])
        b = make_pair(specs_b, hp, seed=7, checked=[])
        load_grads(a, 0, 5)
        load_grads(b, 0, 7)
        torch.cuda.synchronize()
        sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
        if concurrent:
            for _ in range(8):
                a.opt.step(stream=sa)
                b.opt.step(stream=sb)
        else:
            for _ in range(8):
                a.opt.step(stream=sa)
            torch.cuda.synchronize()
            for _ in range(8):
                b.opt.step(stream=sb)
        a.opt.sync_momentum(stream=sa)
        b.opt.sync_momentum(stream=sb)
        torch.cuda.synchronize()
        assert not a.opt.nonfinite() and not b.opt.nonfinite()
        return a, b

    seq = run(False)
    par = run(True)
    for u, v in zip(seq, par):
        for i in range(len(u.specs)):
            assert torch.equal(u.xs[i], v.xs[i]), (u.specs[i].name, "x")
            for k, (su, sv) in enumerate(zip(u.opt.state[i], v.opt.state[i])):
                assert torch.equal(su, sv), (u.specs[i].name, "prc"[k])


def test_deferred_equals_two_pass_bitwise():
    """The deferred half-kick performs the same operations as the two-pass
    schedule, so after syncing the results agree bit for bit."""
    log("[case] deferred vs two-pass")
    a = _run_steps(SPECS_MIX, synth.HP_FRICTION, 7, two_pass=False)
    b = _run_steps(SPECS_MIX, synth.HP_FRICTION, 7, two_pass=True)
    for i in range(len(SPECS_MIX)):
        assert torch.equal(a.xs[i], b.xs[i])
        for u, v in zip(a.opt.state[i], b.opt.state[i]):
            assert torch.equal(u, v)


def test_checkpoint_resume_bitwise():
    """10 steps == 5 steps, sync, save (x, p, r, c), new context on the saved
    state, 5 more steps."""
    log("[case] checkpoint/resume")
    hp = synth.HP_FRICTION
    full = _run_steps(SPECS_MIX, hp, 10)
    first = make_pair(SPECS_MIX, hp, seed=5, checked=[])
    for s in range(5):
        load_grads(first, s, 5)
        first.opt.step()
    first.opt.sync_momentum()
    torch.cuda.synchronize()
    saved_x = [x.clone() for x in first.xs]
    saved_state = [tuple(t.clone() for t in st) for st in first.opt.state]
    first.opt.close()
    gs = [torch.empty_like(x) for x in saved_x]
    opt = R.RIKFAD(saved_x, gs, state=saved_state, **hp)
    first.xs, first.gs, first.opt = saved_x, gs, opt
    for s in range(5, 10):
        load_grads(first, s, 5)
        opt.step()
    opt.sync_momentum()
    torch.cuda.synchronize()
    for i in range(len(SPECS_MIX)):
        assert torch.equal(full.xs[i], saved_x[i])
        for u, v in zip(full.opt.state[i], saved_state[i]):
            assert torch.equal(u, v)


def test_state_changed_after_rewriting_factors():
    """Writing r, c from outside, then rikfad_state_changed, makes the next
    step use the new factor sum (the partial sums of R are rebuilt)."""
    log("[case] state_changed")
    specs = [S("a", 260, 300)]
    hp = synth.HP_FRICTION
    pair = make_pair(specs, hp, seed=6)
    for s in range(3):
        hg = load_grads(pair, s, 6)
        pair.opt.step()
        oracle_step(pair, hg, hp)
    pair.opt.sync_momentum()
    torch.cuda.synchronize()
    o = pair.ref[0]
    p, r, c = pair.opt.state[0]
    r.mul_(3.0)
    c.mul_(0.5)
    o.r[:] = host(r)
    o.c[:] = host(c)
    o.p[:] = host(p)
    o.x[:] = host(pair.xs[0])
    pair.opt.state_changed()
    for s in range(3, 6):
        hg = load_grads(pair, s, 6)
        pair.opt.step()
        oracle_step(pair, hg, hp)
    assert_ok(compare(pair), label="state_changed")


def test_set_hparams_mid_run_applies_pending_kick_first():
    log("[case] set_hparams mid-run")
    specs = [S("a", 200, 260), S("b", 1, 260)]
    hp1 = synth.HP_FRICTION
    hp2 = dict(h=0.05, gamma=0.1, alpha=0.2, mu=0.2, eps_stab=1e-6)
    pair = make_pair(specs, hp1, seed=7)
    for s in range(4):
        hg = load_grads(pair, s, 7)
        pair.opt.step()
        oracle_step(pair, hg, hp1)
    pair.opt.set_hparams(**hp2)
    for s in range(4, 8):
        hg = load_grads(pair, s, 7)
        pair.opt.step()
        oracle_step(pair, hg, hp2)
    assert_ok(compare(pair), label="set_hparams")


def test_step_grads_with_new_buffers():
    """rikfad_step_grads with freshly allocated gradient tensors gives the
    same result as copying into the buffers given at create."""
    log("[case] step_grads")
    hp = synth.HP_FRICTION
    a = _run_steps(SPECS_MIX, hp, 4)
    b = make_pair(SPECS_MIX, hp, seed=5, checked=[])
    for s in range(4):
        new = [torch.from_numpy(b.wl.grad(i, s)).to(b.gs[i].dtype).cuda().contiguous()
               for i in range(len(SPECS_MIX))]
        b.opt.step(grads=new)
    b.opt.sync_momentum()
    torch.cuda.synchronize()
    for i in range(len(SPECS_MIX)):
        assert torch.equal(a.xs[i], b.xs[i])
        for u, v in zip(a.opt.state[i], b.opt.state[i]):
            assert torch.equal(u, v)


def test_step_grads_rejects_misaligned_gradient():
    specs = [S("a", 64, 128)]
    pair = make_pair(specs, synth.HP_BASE, checked=[])
    buf = torch.zeros(64 * 128 + 1, device="cuda")
    with pytest.raises(R.RikfadError) as e:
        pair.opt.step(grads=[buf[1:].view(64, 128)])
    assert e.value.status == R.RIKFAD_EALIGN


def test_nonfinite_gradient_is_flagged_and_propagated():
    log("[case] NaN injection")
    specs = [S("a", 128, 256), S("b", 64, 64)]
    pair = make_pair(specs, synth.HP_BASE, seed=8, checked=[])
    load_grads(pair, 0, 8)
    pair.opt.step()
    assert not pair.opt.nonfinite()
    load_grads(pair, 1, 8)
    pair.gs[0][5, 7] = float("nan")
    pair.opt.step()
    pair.opt.sync_momentum()
    assert pair.opt.nonfinite()
    p, r, c = pair.opt.state[0]
    # the NaN reaches row 5's R, column 7's C and 1^T R, hence every xi~ of
    # this tensor; other tensors are untouched
    assert torch.isnan(r[5]) and torch.isnan(c[7]) and torch.isnan(p).all()
    assert torch.isfinite(c[:7]).all()
    for t in pair.opt.state[1]:
        assert torch.isfinite(t).all()


def test_nonfinite_vector_gradient_is_flagged():
    """A NaN in a bias vector's gradient reaches that entry's element-wise
    friction in the streaming launch, which sets the non-finite flag; the
    other entries and tensors stay finite."""
    log("[case] NaN injection into a vector")
    specs = [S("a", 64, 64), S("v", 1, 300)]
    pair = make_pair(specs, synth.HP_BASE, seed=9, checked=[])
    load_grads(pair, 0, 9)
    pair.opt.step()
    assert not pair.opt.nonfinite()
    load_grads(pair, 1, 9)
    pair.gs[1][0, 17] = float("nan")
    pair.opt.step()
    assert pair.opt.nonfinite()
    _, _, xi = pair.opt.state[1]
    assert torch.isnan(xi[17]) and torch.isfinite(xi[:17]).all() and torch.isfinite(xi[18:]).all()
    for t in pair.opt.state[0]:
        assert torch.isfinite(t).all()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_full_ikfad_flags_nonfinite_friction(dtype):
    log(f"[case] full iKFAD NaN injection {dtype}")
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = (torch.randn((96, 640), device="cuda") * 0.02).to(dt)
    g = torch.randn((96, 640), device="cuda").to(dt)
    ik = R.IKFAD([x], [g], h=0.1, gamma=0.0, alpha=0.1, mu=0.1)
    ik.step()
    assert not ik.nonfinite()
    g[40, 333] = float("inf")
    ik.step()
    assert ik.nonfinite()
    ik.close()


def test_binding_rejects_state_it_cannot_address():
    """The C ABI sees only pointers: the binding refuses caller state that is
    not a contiguous fp32 buffer of the right size on the parameter's device."""
    x = torch.zeros((8, 16), device="cuda")
    g = torch.zeros_like(x)
    good = (torch.zeros((8, 16), device="cuda"), torch.zeros(8, device="cuda"),
            torch.zeros(16, device="cuda"))
    R.RIKFAD([x], [g], h=1e-3, state=[good]).close()
    bad = [
        (torch.zeros((8, 15), device="cuda"), good[1], good[2]),              # short p
        (good[0].double(), good[1], good[2]),                                 # fp64 p
        (torch.zeros((16, 8), device="cuda").t(), good[1], good[2]),          # strided p
        (good[0], torch.zeros(7, device="cuda"), good[2]),                    # short r
        (good[0], good[1], torch.zeros(16)),                                  # host c
    ]
    for st in bad:
        with pytest.raises(ValueError):
            R.RIKFAD([x], [g], h=1e-3, state=[st])
        with pytest.raises(ValueError):
            R.ADAFM([x], [g], h=1e-3, state=[st])
    with pytest.raises(ValueError):
        R.IKFAD([x], [g.double()], h=1e-3)
    with pytest.raises(ValueError):
        R.IKFAD([torch.zeros((16, 8), device="cuda").t()], [g], h=1e-3)


def test_query_reports_state_and_traffic():
    specs = synth.gpt2_small()
    pair = make_pair(specs[:6], synth.HP_BASE, checked=[])
    info = pair.opt.query()
    mats = [s for s in specs[:6] if not s.is_vector]
    vecs = [s for s in specs[:6] if s.is_vector]
    assert info["matrices"] == len(mats) and info["vectors"] == len(vecs)
    assert info["state_bytes"] == sum(4 * s.numel + 4 * (s.m + s.n) for s in mats) + sum(
        8 * s.numel for s in vecs)
    assert info["min_bytes_per_step"] == sum(20 * s.numel + 8 * (s.m + s.n) for s in mats) + sum(
        28 * s.numel for s in vecs)
    pair.opt.step()
    assert pair.opt.query()["pending"] == 1
    pair.opt.sync_momentum()
    assert pair.opt.query()["pending"] == 0


# --------------------------------------------------------- full iKFAD

def _ikfad_parity(specs, hp, steps, seed):
    """Full-tensor iKFAD through the library against the oracle's element-wise
    step; bf16 parameters are reset to the oracle's before every step and
    compared with its unrounded update."""
    wl = synth.Workload(specs, seed=seed)
    dts = [torch.bfloat16 if sp.dtype == "bf16" else torch.float32 for sp in specs]
    xs = [torch.from_numpy(wl.x0(i)).to(dts[i]).cuda() for i in range(len(specs))]
    gs = [torch.empty_like(x) for x in xs]
    ik = R.IKFAD(xs, gs, h=hp["h"], gamma=hp["gamma"], alpha=hp["alpha"], mu=hp["mu"])
    ref = []
    for i in range(len(specs)):
        x = wl.x0(i).astype(np.float64).ravel().copy()
        ref.append((x, np.zeros_like(x), np.zeros_like(x), np.zeros_like(x)))
    for s in range(steps):
        for i, sp in enumerate(specs):
            g = wl.grad(i, s)
            if sp.dtype == "bf16":
                xs[i].copy_(torch.from_numpy(ref[i][0].reshape(xs[i].shape)).to(dts[i]))
            gs[i].copy_(torch.from_numpy(g).to(dts[i]))
            O.ikfad_step(ref[i][0], g.ravel(), ref[i][1], ref[i][2], O.HParams(**hp),
                         x_bf16=(sp.dtype == "bf16"), x_unrounded=ref[i][3])
        ik.step()
        torch.cuda.synchronize()
    for i, sp in enumerate(specs):
        p, xi = ik.state[i]
        bf = sp.dtype == "bf16"
        assert rel_rms(host(xs[i]).ravel(), ref[i][3] if bf else ref[i][0]) < (4e-3 if bf else TOL_F32)
        assert rel_rms(host(p).ravel(), ref[i][1]) < TOL_F32
        assert rel_plain(host(xi).ravel(), ref[i][2]) < TOL_F32


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_full_ikfad_matches_oracle(dtype):
    log(f"[case] full iKFAD {dtype}")
    _ikfad_parity([S("a", 256, 512, dtype), S("b", 1, 100, dtype), S("c", 33, 27, dtype)],
                  synth.HP_FRICTION, 10, seed=9)


@pytest.mark.parametrize("seed", range(6))
def test_full_ikfad_random_sets(seed):
    specs, hp, _ = _random_set(100 + seed)
    log(f"[case] full iKFAD random set seed={100 + seed} hp={hp} "
        f"{[(s.m, s.n, s.dtype) for s in specs]}")
    _ikfad_parity(specs, hp, 5, seed=seed)


# ------------------------------------------------------------- probes

def test_probes_compute_what_they_claim():
    n = 1 << 20
    a, b, c = (torch.randn(n, device="cuda") for _ in range(3))
    d, e = torch.empty_like(a), torch.empty_like(a)
    s = torch.cuda.current_stream().cuda_stream
    R.rikfad_probe_stream(a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), e.data_ptr(),
                          n, s)
    f = torch.empty_like(a)
    R.rikfad_probe_copy(a.data_ptr(), f.data_ptr(), 4 * n, s)
    torch.cuda.synchronize()
    assert torch.equal(d, a + b) and torch.equal(e, a * c) and torch.equal(f, a)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", [0, 1])
def test_mix_probe_computes_what_it_claims(dtype, shape):
    # 1000 rows of 256 elements: several workgroups and a ragged last one
    # in both shapes (4096 and 8192 elements per workgroup).
    n = 256 * 1000
    log(f"[case] probe_mix dtype={dtype} shape={shape} n={n}")
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.randn(n, device="cuda").to(dt)
    g = torch.randn(n, device="cuda").to(dt)
    p = torch.randn(n, device="cuda")
    x0, p0 = x.clone(), p.clone()
    code = R.RIKFAD_BF16 if dtype == "bf16" else R.RIKFAD_FP32
    R.rikfad_probe_mix(x.data_ptr(), g.data_ptr(), p.data_ptr(), n, code, shape,
                       torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    if dtype == "bf16":
        want = x0.view(torch.int16) ^ g.view(torch.int16)
        assert torch.equal(x.view(torch.int16), want)
    else:
        assert torch.equal(x, x0 + g)
    assert torch.equal(p, p0 * 0.5)


def test_write_probe_fills_exactly_its_bytes():
    n = (1 << 20) + 12                      # a ragged last workgroup
    a = torch.zeros(n + 8, device="cuda")
    R.rikfad_probe_write(a.data_ptr(), 4 * n, 0x3f800000,
                         torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.all(a[:n] == 1.0)
    assert torch.all(a[n:] == 0.0)


def test_read_probe_reads_without_writing():
    n = (1 << 20) + 12
    a = torch.randn(n, device="cuda")
    out = torch.full((1,), 7.0, device="cuda")
    R.rikfad_probe_read(a.data_ptr(), 4 * n, out.data_ptr(),
                        torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert out.item() == 7.0

"""Pins of the fp64 Adafactor-m oracle against closed forms and identities.

Adafactor-m (Section 2, Methodology, left-hand system; discrete schedule
beta2_t = 1 - t^{-0.8}, beta1 > 0, no relative step or warm-up, Section 3
and App. "Hyperparameters") is the factored second moment of Shazeer &
Stern (2018) with update clipping and a full first moment.  Each test below
fixes a result by hand (rank-1 gradients make the factored estimate exact,
a diagonal gradient gives a known clipping factor, constant gradients give
geometric first-moment sums), so that a dropped square root, a wrong
schedule exponent, a missing clip or a transposed factor fails one of them.
"""
import math

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _state(m, n, x0=None, mom0=None):
    x = np.zeros((m, n)) if x0 is None else np.array(x0, dtype=np.float64, order="C")
    mom = np.zeros((m, n)) if mom0 is None else np.array(mom0, dtype=np.float64, order="C")
    return x, mom, np.zeros(m), np.zeros(n)


def _rank1_grad(rng, m, n):
    a = rng.uniform(0.5, 2.0, m) * rng.choice([-1.0, 1.0], m)
    b = rng.uniform(0.5, 2.0, n) * rng.choice([-1.0, 1.0], n)
    return np.outer(a, b)


def test_beta2_schedule():
    # beta2_t = 1 - t^{-0.8}: 0 at the first step, then increasing to 1.
    assert oracle.adafm_beta2(1) == 0.0
    assert oracle.adafm_beta2(2) == pytest.approx(1 - 2 ** -0.8, rel=1e-15)
    assert oracle.adafm_beta2(1000) == pytest.approx(1 - 1000 ** -0.8, rel=1e-15)


def test_rank1_gradient_gives_sign_update():
    # For G = a b^T and eps1 = 0 the factored estimate is exact: V = G^2,
    # U = sign(G), RMS(U) = 1 so clipping at d = 1 does nothing.
    rng = np.random.default_rng(1)
    m, n, h, b1 = 5, 7, 0.01, 0.9
    g = _rank1_grad(rng, m, n)
    x0 = rng.standard_normal((m, n))
    x, mom, r, c = _state(m, n, x0)
    hp = oracle.AdafmHParams(h=h, beta1=b1, eps1=0.0)
    oracle.adafm_matrix_step(x, g, mom, r, c, 1, hp)
    np.testing.assert_allclose(mom, (1 - b1) * h * np.sign(g), rtol=1e-14, atol=0)
    np.testing.assert_allclose(x, x0 - (1 - b1) * h * np.sign(g), rtol=1e-14, atol=1e-17)
    np.testing.assert_allclose(r, (g * g).sum(1), rtol=1e-14)
    np.testing.assert_allclose(c, (g * g).sum(0), rtol=1e-14)


def test_constant_gradient_first_moment_geometric_sum():
    # Constant rank-1 G: the second-moment factors stay at the row/column
    # sums of G^2 (every beta2_t average of a constant), U = sign(G) each
    # step, M_t = h sign(G) (1 - beta1^t), X_t = X_0 - h sign(G) sum_k (1 - beta1^k).
    rng = np.random.default_rng(2)
    m, n, h, b1, T = 4, 6, 0.003, 0.8, 7
    g = _rank1_grad(rng, m, n)
    x0 = rng.standard_normal((m, n))
    x, mom, r, c = _state(m, n, x0)
    hp = oracle.AdafmHParams(h=h, beta1=b1, eps1=0.0)
    for t in range(1, T + 1):
        oracle.adafm_matrix_step(x, g, mom, r, c, t, hp)
        np.testing.assert_allclose(mom, h * np.sign(g) * (1 - b1 ** t), rtol=1e-13)
    drift = sum(1 - b1 ** k for k in range(1, T + 1))
    np.testing.assert_allclose(x, x0 - h * np.sign(g) * drift, rtol=1e-13, atol=1e-16)


@pytest.mark.parametrize("d, div", [(1.0, 1.25), (0.5, 2.5), (2.0, 1.0), (0.0, 1.0)])
def test_clipping_closed_form(d, div):
    # G = diag(1, 2), eps1 = 0: R = C = (1, 4), 1^T R = 5, so
    # U_11 = 1 / sqrt(1/5) = sqrt(5), U_22 = 2 / sqrt(16/5) = sqrt(5)/2, and
    # RMS(U) = sqrt((5 + 5/4) / 4) = 1.25.  Clipping divides by max(1, 1.25/d).
    g = np.array([[1.0, 0.0], [0.0, 2.0]])
    h, b1 = 0.01, 0.9
    x, mom, r, c = _state(2, 2)
    hp = oracle.AdafmHParams(h=h, beta1=b1, eps1=0.0, clip_threshold=d)
    oracle.adafm_matrix_step(x, g, mom, r, c, 1, hp)
    u = np.array([[math.sqrt(5.0), 0.0], [0.0, math.sqrt(5.0) / 2]])
    np.testing.assert_allclose(mom, (1 - b1) * h * u / div, rtol=1e-14, atol=0)
    np.testing.assert_allclose(x, -(1 - b1) * h * u / div, rtol=1e-14, atol=0)
    np.testing.assert_allclose(r, [1.0, 4.0], rtol=1e-15)
    np.testing.assert_allclose(c, [1.0, 4.0], rtol=1e-15)


def test_second_step_uses_schedule():
    # G_1 = 1 (2x2), G_2 = 2 (2x2), eps1 = 0, no clipping.  Step 1: R = C = 2,
    # U = 1.  Step 2 with b = 1 - 2^{-0.8}: R = C = 2b + 8(1-b) = 8 - 6b,
    # V = (8 - 6b)^2 / (2 (8 - 6b)) = 4 - 3b, U = 2 / sqrt(4 - 3b).
    h, b1 = 0.02, 0.7
    b = 1 - 2 ** -0.8
    x, mom, r, c = _state(2, 2)
    hp = oracle.AdafmHParams(h=h, beta1=b1, eps1=0.0, clip_threshold=0.0)
    oracle.adafm_matrix_step(x, np.ones((2, 2)), mom, r, c, 1, hp)
    np.testing.assert_allclose(mom, (1 - b1) * h, rtol=1e-15)
    oracle.adafm_matrix_step(x, 2 * np.ones((2, 2)), mom, r, c, 2, hp)
    u2 = 2 / math.sqrt(4 - 3 * b)
    m2 = b1 * (1 - b1) * h + (1 - b1) * h * u2
    np.testing.assert_allclose(r, 8 - 6 * b, rtol=1e-14)
    np.testing.assert_allclose(c, 8 - 6 * b, rtol=1e-14)
    np.testing.assert_allclose(mom, m2, rtol=1e-14)
    np.testing.assert_allclose(x, -((1 - b1) * h + m2), rtol=1e-14)


def test_parameter_scale():
    # a_t = h max(eps2, RMS(X_{t-1})): X_0 = 0.5 everywhere halves the step;
    # X_0 = 0 gives h * eps2.
    rng = np.random.default_rng(3)
    m, n, h, b1 = 3, 4, 0.01, 0.9
    g = _rank1_grad(rng, m, n)
    hp = oracle.AdafmHParams(h=h, beta1=b1, eps1=0.0, scale_parameter=True, eps2=1e-3)
    x, mom, r, c = _state(m, n, np.full((m, n), 0.5))
    oracle.adafm_matrix_step(x, g, mom, r, c, 1, hp)
    np.testing.assert_allclose(x, 0.5 - (1 - b1) * h * 0.5 * np.sign(g), rtol=1e-14)
    x, mom, r, c = _state(m, n)
    oracle.adafm_matrix_step(x, g, mom, r, c, 1, hp)
    np.testing.assert_allclose(x, -(1 - b1) * h * 1e-3 * np.sign(g), rtol=1e-14)


def test_zero_gradient_eps1_and_zero_estimate():
    # G = 0: R = n eps1, C = m eps1 after the first step, U = 0, so only the
    # first-moment decay moves X.  With eps1 = 0 as well the estimate is 0
    # and U is taken as 0 (no 0/0).
    m, n, b1 = 3, 5, 0.6
    rng = np.random.default_rng(4)
    mom0 = rng.standard_normal((m, n))
    x0 = rng.standard_normal((m, n))
    for eps1 in (1e-3, 0.0):
        x, mom, r, c = _state(m, n, x0, mom0)
        hp = oracle.AdafmHParams(h=0.1, beta1=b1, eps1=eps1)
        oracle.adafm_matrix_step(x, np.zeros((m, n)), mom, r, c, 1, hp)
        np.testing.assert_allclose(r, n * eps1, rtol=1e-15)
        np.testing.assert_allclose(c, m * eps1, rtol=1e-15)
        np.testing.assert_allclose(mom, b1 * mom0, rtol=1e-15)
        np.testing.assert_allclose(x, x0 - b1 * mom0, rtol=1e-15)
        assert np.isfinite(x).all()


def test_transpose_invariance():
    # The factored estimate is symmetric in rows and columns: stepping the
    # transposed problem gives the transposed state with R and C swapped.
    rng = np.random.default_rng(5)
    m, n = 5, 3
    hp = oracle.AdafmHParams(h=0.01, beta1=0.9)
    x0 = rng.standard_normal((m, n))
    xa, ma, ra, ca = _state(m, n, x0)
    xb, mb, rb, cb = _state(n, m, x0.T)
    for t in range(1, 5):
        g = rng.standard_normal((m, n)) * rng.uniform(0.1, 3.0, (m, 1))
        oracle.adafm_matrix_step(xa, g, ma, ra, ca, t, hp)
        oracle.adafm_matrix_step(xb, np.ascontiguousarray(g.T), mb, rb, cb, t, hp)
    np.testing.assert_allclose(xb, xa.T, rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(mb, ma.T, rtol=1e-13, atol=1e-18)
    np.testing.assert_allclose(rb, ca, rtol=1e-13)
    np.testing.assert_allclose(cb, ra, rtol=1e-13)


def test_gradient_scale_invariance():
    # With eps1 = 0 the update G / sqrt(V) does not change when G is scaled;
    # the factors scale with its square.
    rng = np.random.default_rng(6)
    m, n = 6, 4
    hp = oracle.AdafmHParams(h=0.01, beta1=0.9, eps1=0.0)
    x0 = rng.standard_normal((m, n))
    xa, ma, ra, ca = _state(m, n, x0)
    xb, mb, rb, cb = _state(m, n, x0)
    for t in range(1, 4):
        g = rng.standard_normal((m, n))
        oracle.adafm_matrix_step(xa, g, ma, ra, ca, t, hp)
        oracle.adafm_matrix_step(xb, 1000.0 * g, mb, rb, cb, t, hp)
    np.testing.assert_allclose(xb, xa, rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(mb, ma, rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(rb, 1e6 * ra, rtol=1e-13)


@pytest.mark.parametrize("shape", [(1, 9), (9, 1)])
def test_vector_matches_factored_single_row_or_column(shape):
    # A 1 x n (or n x 1) matrix: the factored estimate R C^T / 1^T R equals
    # the unfactored second moment (C for one row, R for one column).
    rng = np.random.default_rng(7)
    m, n = shape
    k = m * n
    hp = oracle.AdafmHParams(h=0.01, beta1=0.9)
    x0 = rng.standard_normal((m, n))
    xa, ma, ra, ca = _state(m, n, x0)
    xv = x0.reshape(-1).copy()
    mv = np.zeros(k)
    v = np.zeros(k)
    for t in range(1, 5):
        g = rng.standard_normal((m, n))
        oracle.adafm_matrix_step(xa, g, ma, ra, ca, t, hp)
        oracle.adafm_vector_step(xv, g.reshape(-1), mv, v, t, hp)
    np.testing.assert_allclose(xv, xa.reshape(-1), rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(mv, ma.reshape(-1), rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(v, (ca if m == 1 else ra), rtol=1e-13)


def test_vector_constant_gradient_closed_form():
    # Unfactored: constant g keeps v = g^2 (eps1 = 0), U = sign(g).
    h, b1, T = 0.01, 0.75, 5
    g = np.array([0.5, -2.0, 3.0, -0.25])
    x = np.zeros(4)
    mom = np.zeros(4)
    v = np.zeros(4)
    hp = oracle.AdafmHParams(h=h, beta1=b1, eps1=0.0)
    for t in range(1, T + 1):
        oracle.adafm_vector_step(x, g, mom, v, t, hp)
    np.testing.assert_allclose(v, g * g, rtol=1e-15)
    np.testing.assert_allclose(mom, h * np.sign(g) * (1 - b1 ** T), rtol=1e-14)
    drift = sum(1 - b1 ** k for k in range(1, T + 1))
    np.testing.assert_allclose(x, -h * np.sign(g) * drift, rtol=1e-14)


def test_bf16_storage_rounds_unrounded_update():
    # bf16 parameters: x_unrounded = X - M before rounding, X = its nearest bf16.
    rng = np.random.default_rng(8)
    m, n = 4, 8
    x0 = oracle.round_bf16(rng.standard_normal((m, n)))
    x, mom, r, c = _state(m, n, x0)
    xu = np.zeros((m, n))
    hp = oracle.AdafmHParams(h=0.05, beta1=0.9)
    oracle.adafm_matrix_step(x, rng.standard_normal((m, n)), mom, r, c, 1, hp,
                             x_bf16=True, x_unrounded=xu)
    np.testing.assert_array_equal(xu, x0 - mom)
    np.testing.assert_array_equal(x, oracle.round_bf16(xu))


def test_step_list_dispatch():
    # The list entry point runs the factored step on matrices and the
    # unfactored one on vectors, with v in c (m == 1) or r (n == 1).
    rng = np.random.default_rng(9)
    hp = oracle.AdafmHParams(h=0.01, beta1=0.9)
    shapes = [(3, 5), (1, 6), (4, 1)]
    ts = [oracle.make_tensor(rng.standard_normal(s)) for s in shapes]
    ref = [oracle.make_tensor(t.x) for t in ts]
    for t in range(1, 3):
        gs = [rng.standard_normal(s) for s in shapes]
        oracle.adafm_step_list(ts, gs, t, hp, threads=2)
        oracle.adafm_matrix_step(ref[0].x, gs[0], ref[0].p, ref[0].r, ref[0].c, t, hp)
        oracle.adafm_vector_step(ref[1].x.reshape(-1), gs[1].reshape(-1), ref[1].p.reshape(-1),
                                 ref[1].c, t, hp)
        oracle.adafm_vector_step(ref[2].x.reshape(-1), gs[2].reshape(-1), ref[2].p.reshape(-1),
                                 ref[2].r, t, hp)
    for a, b in zip(ts, ref):
        np.testing.assert_array_equal(a.x, b.x)
        np.testing.assert_array_equal(a.p, b.p)
        np.testing.assert_array_equal(a.xi if a.is_vector else a.r, b.xi if b.is_vector else b.r)


def test_rejects_bad_arguments():
    x, mom, r, c = _state(2, 2)
    g = np.ones((2, 2))
    with pytest.raises(RuntimeError):
        oracle.adafm_matrix_step(x, g, mom, r, c, 0, oracle.AdafmHParams(h=0.1))
    with pytest.raises(RuntimeError):
        oracle.adafm_matrix_step(x, g, mom, r, c, 1, oracle.AdafmHParams(h=0.1, beta1=1.0))
    with pytest.raises(RuntimeError):
        oracle.adafm_matrix_step(x, g, mom, r, c, 1, oracle.AdafmHParams(h=0.1, decay_rate=0.5))

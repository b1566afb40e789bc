"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each test checks the oracle against a different route to the same value:
an SVD closed form, the textbook cubic iteration's limit (the polar factor),
hand-worked fixtures under ``tests/golden/``, special cases and invariants
that the paper states (Algorithm 1, Table 1, Appendix F). A plausible slip in
the oracle (a dropped term, a wrong sign or index, a transposed operand, the
post-update momentum in the interpolation, swapped betas) fails at least one.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import lionmuon_oracle as lo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _scalar_iterate(x, coeffs, steps):
    """The scalar odd polynomial(s) applied ``steps`` times to singular
    values; ``coeffs`` is one (a, b, c) or a list of per-step triples."""
    sched = [coeffs] * steps if np.ndim(coeffs) == 1 else list(coeffs)
    assert len(sched) == steps
    for a, b, c in sched:
        x = a * x + b * x ** 3 + c * x ** 5
    return x


def _svd_closed_form(G, steps, coeffs, eps):
    """NS_K(G) = U diag(p^K(sigma_i / (||G||_F + eps))) V^T.

    An odd matrix polynomial of the form a X + b (X X^T) X + c (X X^T)^2 X
    keeps the singular vectors and maps each singular value through the
    scalar polynomial; ||G||_F is taken from the singular values.
    """
    U, s, Vt = np.linalg.svd(np.asarray(G, np.float64), full_matrices=False)
    fro = np.sqrt(np.sum(s ** 2))
    x = s / (fro + eps)
    return (U * _scalar_iterate(x, coeffs, steps)) @ Vt


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# --------------------------------------------------------------------------
# Newton-Schulz
# --------------------------------------------------------------------------
def test_quintic_coefficients_match_published_values():
    g = _golden("ns_quintic_coefficients.json")
    assert oracle.QUINTIC == (g["a"], g["b"], g["c"])
    cub = g["cubic_textbook"]
    assert oracle.CUBIC == (cub["a"], cub["b"], cub["c"])
    assert oracle.NS_STEPS == 5  # Table 3


@pytest.mark.parametrize("shape", [(2, 3), (3, 2), (5, 7), (7, 5), (32, 48),
                                   (48, 32), (64, 64), (96, 40), (1, 9), (9, 1)])
@pytest.mark.parametrize("eps", [0.0, 1e-7])
def test_ns_matches_svd_closed_form(shape, eps):
    rng = np.random.default_rng([11, *shape])
    G = rng.standard_normal(shape) * 1e-2
    got = oracle.newton_schulz(G, 5, oracle.QUINTIC, eps)
    ref = _svd_closed_form(G, 5, oracle.QUINTIC, eps)
    assert got.shape == G.shape
    assert _rel(got, ref) < 1e-11


@pytest.mark.parametrize("steps", [0, 1, 2, 3, 7])
def test_ns_step_count_matches_closed_form(steps):
    rng = np.random.default_rng(5)
    G = rng.standard_normal((12, 20))
    got = oracle.newton_schulz(G, steps, oracle.QUINTIC, 1e-7)
    ref = _svd_closed_form(G, steps, oracle.QUINTIC, 1e-7)
    assert _rel(got, ref) < 1e-12


SCHEDULES = {
    "quintic3_cubic2": [oracle.QUINTIC] * 3 + [oracle.CUBIC] * 2,
    "decreasing": [(3.0, -3.2, 1.2), (2.5, -2.0, 0.5), (2.0, -1.3, 0.3), (1.7, -0.8, 0.1),
                   (1.5, -0.5, 0.0)],
}


@pytest.mark.parametrize("name", sorted(SCHEDULES))
@pytest.mark.parametrize("shape", [(6, 9), (40, 24), (64, 64)])
def test_ns_per_step_schedule_matches_closed_form(name, shape):
    """Section 2: other odd-polynomial schedules (per-step coefficients) share
    the cost structure; the oracle takes one triple per step."""
    rng = np.random.default_rng([31, *shape])
    G = rng.standard_normal(shape)
    sched = SCHEDULES[name]
    got = oracle.newton_schulz(G, 5, sched, 1e-7)
    assert _rel(got, _svd_closed_form(G, 5, sched, 1e-7)) < 1e-12
    # a constant schedule equals the single-triple form
    assert np.array_equal(oracle.newton_schulz(G, 5, [oracle.QUINTIC] * 5),
                          oracle.newton_schulz(G, 5, oracle.QUINTIC))
    with pytest.raises(ValueError):
        oracle.newton_schulz(G, 4, sched)


@pytest.mark.parametrize("shape", [(3, 5), (6, 4), (8, 8)])
def test_cubic_iteration_converges_to_polar_factor(shape):
    """Textbook reduction: the cubic NS iteration converges to U V^T."""
    rng = np.random.default_rng(sum(shape))
    k = min(shape)
    U, _ = np.linalg.qr(rng.standard_normal((shape[0], k)))
    V, _ = np.linalg.qr(rng.standard_normal((shape[1], k)))
    sig = np.linspace(1.0, 3.0, k)
    G = (U * sig) @ V.T
    got = oracle.newton_schulz(G, 40, oracle.CUBIC, 0.0)
    assert np.max(np.abs(got - U @ V.T)) < 1e-10


def test_rank_one_maps_to_scaled_outer_product():
    rng = np.random.default_rng(3)
    u, v = rng.standard_normal(17), rng.standard_normal(29)
    G = np.outer(u, v)
    gain = _scalar_iterate(1.0, oracle.QUINTIC, 5)
    assert abs(gain - 0.6964) < 5e-4            # p^5(1) of the quintic
    ref = gain * np.outer(u / np.linalg.norm(u), v / np.linalg.norm(v))
    assert _rel(oracle.newton_schulz(G, 5, oracle.QUINTIC, 0.0), ref) < 1e-12
    # eps shifts the normalised singular value by a relative ~eps/||G||.
    assert _rel(oracle.newton_schulz(G, 5, oracle.QUINTIC, 1e-7), ref) < 1e-6


def test_orthonormal_rows_map_to_scaled_copy():
    rng = np.random.default_rng(4)
    m, n = 4, 10
    Q, _ = np.linalg.qr(rng.standard_normal((n, m)))
    Q = Q.T                                       # m x n, orthonormal rows
    gain = _scalar_iterate(1.0 / np.sqrt(m), oracle.QUINTIC, 5)
    assert abs(gain - 0.76544) < 1e-4             # p^5(1/2)
    got = oracle.newton_schulz(Q, 5, oracle.QUINTIC, 0.0)
    assert np.max(np.abs(got - gain * Q)) < 1e-12


def test_zero_input_maps_to_zero_and_sign_zero_is_zero():
    assert np.all(oracle.newton_schulz(np.zeros((6, 9))) == 0.0)
    s = oracle.elementwise_sign(np.array([-0.0, 0.0, 3.0, -2e-30]))
    assert list(s) == [0.0, 0.0, 1.0, -1.0]


def test_transpose_invariance():
    rng = np.random.default_rng(8)
    G = rng.standard_normal((40, 70))
    a = oracle.newton_schulz(G)
    b = oracle.newton_schulz(G.T).T
    assert _rel(a, b) < 1e-12


def test_ns_scale_invariance():
    rng = np.random.default_rng(9)
    G = rng.standard_normal((30, 50))
    a = oracle.newton_schulz(G, eps=0.0)
    b = oracle.newton_schulz(7.5e-4 * G, eps=0.0)
    assert _rel(a, b) < 1e-12


def test_band_of_five_quintic_steps():
    """Singular values of NS_5 output lie in [0.6818, 1.2024] wherever the
    normalised input singular value is >= 1.6e-3 (from the scalar map; at
    1.5e-3 the fifth iterate is still 0.6798)."""
    xs = np.concatenate([np.geomspace(1.6e-3, 1.0, 20000), [1.0]])
    ys = _scalar_iterate(xs, oracle.QUINTIC, 5)
    assert ys.min() >= 0.6818 - 1e-4 and ys.max() <= 1.2024 + 1e-4
    rng = np.random.default_rng(10)
    G = rng.standard_normal((128, 192))
    s_in = np.linalg.svd(G, compute_uv=False)
    x = s_in / np.sqrt(np.sum(s_in ** 2))
    out = oracle.newton_schulz(G)
    s_out = np.linalg.svd(out, compute_uv=False)
    sel = x >= 1.6e-3
    assert sel.sum() > 100
    # singular values are sorted the same way (p^5 is increasing on [0, 0.4])
    assert s_out[sel].min() >= 0.6818 - 1e-6 and s_out.max() <= 1.2024 + 1e-6


def test_ns_differs_from_exact_msign_but_stays_close():
    """The specified result is NS_5, not U V^T: on a Gaussian square matrix the
    two differ by a few tenths in relative Frobenius norm."""
    rng = np.random.default_rng(12)
    G = rng.standard_normal((64, 64))
    U, _, Vt = np.linalg.svd(G)
    d = _rel(oracle.newton_schulz(G), U @ Vt)
    assert 0.05 < d < 0.4


def test_output_scale_rms02():
    assert oracle.ns_output_scale(768, 3072, oracle.SCALE_RMS02) == pytest.approx(
        0.2 * np.sqrt(3072))
    assert oracle.ns_output_scale(5, 3, oracle.SCALE_NONE) == 1.0
    rng = np.random.default_rng(13)
    W = rng.standard_normal((6, 10)) * 0.02
    G = rng.standard_normal((6, 10))
    M = np.zeros_like(G)
    w1, _ = oracle.lionmuon_update(W, G, M, 0, 1, 0.9, 0.99, 0.1, 0.1, 0.0,
                                   scale_mode=oracle.SCALE_RMS02)
    w0, _ = oracle.lionmuon_update(W, G, M, 0, 1, 0.9, 0.99, 0.1, 0.1, 0.0)
    kappa = 0.2 * np.sqrt(10)
    assert _rel(W - w1, kappa * (W - w0)) < 1e-12


# --------------------------------------------------------------------------
# Algorithm 1: branch rule, Lion step, momentum, weight decay
# --------------------------------------------------------------------------
def test_branch_rule():
    assert [oracle.is_muon_step(t, 2) for t in range(5)] == [True, False, True, False, True]
    assert all(oracle.is_muon_step(t, 1) for t in range(6))
    assert not any(oracle.is_muon_step(t, 0) for t in range(50))   # P = infinity
    assert [oracle.is_muon_step(t, 3) for t in range(1, 7)] == [False, False, True,
                                                                False, False, True]
    with pytest.raises(ValueError):
        oracle.is_muon_step(-1, 2)


def test_pure_lion_never_calls_newton_schulz(monkeypatch):
    def boom(*a, **k):
        raise AssertionError("Newton-Schulz called with P = infinity")
    monkeypatch.setattr(lo, "newton_schulz", boom)
    rng = np.random.default_rng(1)
    W, G, M = (rng.standard_normal((8, 8)) for _ in range(3))
    for t in range(4):
        W, M = lo.lionmuon_update(W, G, M, t, 0, 0.9, 0.99, 1e-3, 1e-3, 0.1)


def test_hand_worked_lion_step():
    g = _golden("lion_interpolation_example.json")
    W, M, G = (np.array(g[k]) for k in ("W", "M", "G"))
    w, m = oracle.lionmuon_update(W, G, M, g["t"], g["P"], g["beta1"], g["beta2"],
                                  99.0, g["lr"], g["wd"])
    assert np.allclose(w, g["expected_W"], atol=1e-15, rtol=0)
    assert np.allclose(m, g["expected_M"], atol=1e-15, rtol=0)
    # sign pattern recovered from the step
    sign = -(w - W * (1 - g["lr"] * g["wd"])) / g["lr"]
    assert np.allclose(sign, g["expected_sign"], atol=1e-12)


def test_lion_step_from_zero_momentum():
    rng = np.random.default_rng(2)
    W = rng.standard_normal((5, 6))
    G = rng.standard_normal((5, 6))
    G[0, 0] = 0.0
    M = np.zeros_like(G)
    lr, wd, b1, b2 = 0.01, 0.1, 0.9, 0.99
    w, m = oracle.lionmuon_update(W, G, M, 1, 2, b1, b2, 123.0, lr, wd)
    for i in range(5):
        for j in range(6):
            s = 1.0 if G[i, j] > 0 else (-1.0 if G[i, j] < 0 else 0.0)
            assert w[i, j] == pytest.approx(W[i, j] - lr * (s + wd * W[i, j]), abs=1e-15)
            assert m[i, j] == pytest.approx((1 - b2) * G[i, j], abs=1e-18)


def test_muon_branch_uses_interpolated_direction_and_muon_lr():
    rng = np.random.default_rng(14)
    W = rng.standard_normal((12, 20)) * 0.02
    G = rng.standard_normal((12, 20))
    M = rng.standard_normal((12, 20))
    lr_m, wd, b1 = 0.03, 0.1, 0.9
    w, _ = oracle.lionmuon_update(W, G, M, 4, 2, b1, 0.99, lr_m, 9.0, wd)
    direction = _svd_closed_form(b1 * M + (1 - b1) * G, 5, oracle.QUINTIC, 1e-7)
    assert _rel(w, W - lr_m * (direction + wd * W)) < 1e-12


def test_decoupled_weight_decay_alone():
    """G = M = 0: both branches reduce to W <- (1 - eta*lambda) W."""
    W = np.random.default_rng(6).standard_normal((7, 9))
    Z = np.zeros_like(W)
    w_muon, m1 = oracle.lionmuon_update(W, Z, Z, 0, 1, 0.9, 0.99, 0.3, 0.7, 0.1)
    w_lion, m2 = oracle.lionmuon_update(W, Z, Z, 1, 2, 0.9, 0.99, 0.3, 0.7, 0.1)
    assert np.allclose(w_muon, (1 - 0.03) * W, rtol=0, atol=1e-15)
    assert np.allclose(w_lion, (1 - 0.07) * W, rtol=0, atol=1e-15)
    assert not m1.any() and not m2.any()


def test_update_is_invariant_to_gradient_scale():
    """sign and msign are positively homogeneous of degree zero (Appendix F):
    scaling (G, M) by c > 0 leaves the weight update unchanged."""
    rng = np.random.default_rng(15)
    W = rng.standard_normal((10, 14)) * 0.02
    G = rng.standard_normal((10, 14))
    M = rng.standard_normal((10, 14))
    for t in (0, 1):
        w1, m1 = oracle.lionmuon_update(W, G, M, t, 2, 0.9, 0.99, 0.02, 0.02, 0.1, eps=0.0)
        w2, m2 = oracle.lionmuon_update(W, 50 * G, 50 * M, t, 2, 0.9, 0.99, 0.02, 0.02,
                                        0.1, eps=0.0)
        assert _rel(w1, w2) < 1e-12
        assert _rel(50 * m1, m2) < 1e-14


def test_signmuon_direction_is_updated_ema():
    """Table 1: beta1 = beta2 gives SignMuon / Signum; the interpolation then
    equals this step's updated EMA buffer."""
    rng = np.random.default_rng(16)
    W = rng.standard_normal((6, 6))
    G = rng.standard_normal((6, 6))
    M = rng.standard_normal((6, 6))
    beta, lr = 0.9, 0.05
    w, m = oracle.lionmuon_update(W, G, M, 1, 0, beta, beta, 1.0, lr, 0.0)
    assert np.allclose(w, W - lr * np.sign(m), atol=1e-15)


def test_heavy_ball_and_ema_give_same_iterates():
    """Appendix F: with mu = beta, the EMA buffer is (1-beta) times the
    heavy-ball buffer, so both produce the same directions and, with lambda = 0,
    the same iterates (sign exactly; NS up to the eps guard)."""
    rng = np.random.default_rng(17)
    beta, lr, P = 0.9, 0.01, 2
    W_ema = rng.standard_normal((8, 12)) * 0.02
    W_hb = W_ema.copy()
    M_ema = np.zeros_like(W_ema)
    M_hb = np.zeros_like(W_ema)
    for t in range(6):
        G = rng.standard_normal(W_ema.shape)
        W_ema, M_ema = oracle.lionmuon_update(W_ema, G, M_ema, t, P, beta, beta, lr, lr,
                                              0.0, eps=0.0)
        M_hb = beta * M_hb + G
        if t % P == 0:
            d = oracle.newton_schulz(M_hb, eps=0.0)
        else:
            d = oracle.elementwise_sign(M_hb)
        W_hb = W_hb - lr * d
        assert np.allclose(M_ema, (1 - beta) * M_hb, rtol=1e-12, atol=1e-15)
        assert _rel(W_ema, W_hb) < 1e-12


def test_one_dimensional_and_lion_only_tensors_take_lion_branch():
    rng = np.random.default_rng(18)
    vec = rng.standard_normal((1, 9))
    mat = rng.standard_normal((4, 9))
    Z = np.zeros_like(mat)
    lr = 0.1
    out_w, _ = oracle.lionmuon_step([vec, mat, mat], [vec, mat, mat],
                                    [np.zeros_like(vec), Z, Z], 0, 1, 0.9, 0.99,
                                    5.0, lr, 0.0, lion_only=[False, True, False])
    assert np.allclose(out_w[0], vec - lr * np.sign(vec))
    assert np.allclose(out_w[1], mat - lr * np.sign(mat))
    assert not np.allclose(out_w[2], mat - lr * np.sign(mat))


def test_stable_rank_estimate():
    rng = np.random.default_rng(19)
    u, v = rng.standard_normal(10), rng.standard_normal(7)
    assert oracle.stable_rank_estimate(np.outer(u, v)) == pytest.approx(1.0, rel=1e-12)
    assert oracle.stable_rank_estimate(np.eye(6)) == pytest.approx(6.0, rel=1e-12)
    G = rng.standard_normal((20, 30))
    s = np.linalg.svd(G, compute_uv=False)
    assert oracle.stable_rank_estimate(G, power_steps=500) == pytest.approx(
        np.sum(s ** 2) / s[0] ** 2, rel=1e-8)
    assert oracle.stable_rank_estimate(np.zeros((3, 4))) == 0.0


# --------------------------------------------------------------------------
# AdamW fallback for 1-D parameters (Section 3, implementation notes; Table 3)
# --------------------------------------------------------------------------
def test_adamw_first_step_is_independent_of_betas():
    """At step 1 from zero moments, bias correction gives mhat = g and
    vhat = g^2 exactly, whatever the betas."""
    rng = np.random.default_rng(40)
    W, G = rng.standard_normal(50), rng.standard_normal(50)
    G[3] = 0.0
    Z = np.zeros(50)
    lr, eps, wd = 1e-3, 1e-8, 0.05
    expect = W - lr * (G / (np.abs(G) + eps) + wd * W)
    for b1, b2 in [(0.8, 0.999), (0.9, 0.95), (0.0, 0.5)]:
        w, m, v = oracle.adamw_update(W, G, Z, Z, 1, lr, b1, b2, eps, wd)
        assert np.allclose(w, expect, rtol=0, atol=1e-15)
        assert np.allclose(m, (1 - b1) * G) and np.allclose(v, (1 - b2) * G ** 2)


def test_adamw_constant_gradient_gives_unit_steps():
    """With a constant gradient the bias-corrected moments equal g and g^2
    exactly at every step, so each update is lr * g / (|g| + eps)."""
    g = np.array([0.3, -2.0, 1e-3, 5.0])
    W = np.array([0.1, 0.2, -0.3, 0.4])
    m = v = np.zeros(4)
    lr, eps = 1e-3, 1e-8
    for step in range(1, 8):
        w_new, m, v = oracle.adamw_update(W, g, m, v, step, lr, 0.8, 0.999, eps, 0.0)
        assert np.allclose(W - w_new, lr * g / (np.abs(g) + eps), rtol=1e-12, atol=0)
        W = w_new


def test_adamw_scale_invariance_and_zero_gradient():
    rng = np.random.default_rng(41)
    W, G1, G2 = rng.standard_normal(20), rng.standard_normal(20), rng.standard_normal(20)
    Z = np.zeros(20)
    a = oracle.adamw_update(W, G1, Z, Z, 1, 1e-3, 0.8, 0.999, 0.0, 0.0)
    a = oracle.adamw_update(a[0], G2, a[1], a[2], 2, 1e-3, 0.8, 0.999, 0.0, 0.0)
    b = oracle.adamw_update(W, 7 * G1, Z, Z, 1, 1e-3, 0.8, 0.999, 0.0, 0.0)
    b = oracle.adamw_update(b[0], 7 * G2, b[1], b[2], 2, 1e-3, 0.8, 0.999, 0.0, 0.0)
    assert _rel(a[0], b[0]) < 1e-13
    w, m, v = oracle.adamw_update(W, Z, Z, Z, 3, 1e-3, 0.8, 0.999, 1e-8, 0.1)
    assert np.allclose(w, W * (1 - 1e-4), rtol=1e-15, atol=0)
    with pytest.raises(ValueError):
        oracle.adamw_update(W, G1, Z, Z, 0, 1e-3, 0.8, 0.999, 1e-8, 0.0)


# --------------------------------------------------------------------------
# Adaptive Muon / Lion selection by stable rank (Appendix G)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("shape", [(12, 20), (20, 12), (9, 9)])
def test_stable_rank_power_iteration_closed_form(shape):
    """With S the short-side view (M, or M^T for wide M), singular values sigma,
    and c_i the start vector's components along S's right singular vectors V
    (square, so nothing of v0 lies outside their span), k power steps give v_k
    proportional to V diag(sigma^(2k)) c and sigma_hat^2 = sum (sigma_i coef_i)^2
    / sum coef_i^2 with coef = sigma^(2k) c."""
    rng = np.random.default_rng(42)
    m, n = shape
    s, l = min(m, n), max(m, n)
    U, _ = np.linalg.qr(rng.standard_normal((l, l)))
    V, _ = np.linalg.qr(rng.standard_normal((s, s)))
    sig = np.linspace(3.0, 0.5, s)
    S = (U[:, :s] * sig) @ V.T                      # l x s, singular values sig
    M = S.T if m < n else S
    c = V.T @ (np.ones(s) / np.sqrt(s))
    for k in (0, 1, 3, 8):
        coef = sig ** (2 * k) * c
        sigma_hat2 = np.sum((sig * coef) ** 2) / np.sum(coef ** 2)
        expect = np.sum(sig ** 2) / sigma_hat2
        assert oracle.stable_rank_estimate(M, k) == pytest.approx(expect, rel=1e-12)
    # a start vector along the top singular direction is exact at once
    assert oracle.stable_rank_estimate(M, 0, v0=V[:, 0]) == pytest.approx(
        np.sum(sig ** 2) / sig[0] ** 2, rel=1e-12)


def test_stable_rank_degenerate_iterates():
    """A start vector in the null space of S gives a vanishing iterate: the
    estimate is 0, as for the zero matrix."""
    M = np.array([[1.0, -1.0], [2.0, -2.0], [3.0, -3.0]])   # tall, S = M, v0 = ones
    assert oracle.stable_rank_estimate(M, 0) == 0.0
    assert oracle.stable_rank_estimate(M, 3) == 0.0
    assert oracle.stable_rank_estimate(M.T, 3) == 0.0        # wide: S = M^T = M
    assert oracle.stable_rank_estimate(M, 3, v0=np.array([1.0, 0.0])) == pytest.approx(1.0)


def test_adaptive_rule_threshold_and_branches():
    rng = np.random.default_rng(43)
    m, n = 30, 50
    u, v = rng.standard_normal(m), rng.standard_normal(n)
    low = np.outer(u, v) + 1e-3 * rng.standard_normal((m, n))     # stable rank ~ 1
    high = rng.standard_normal((m, n))                             # stable rank >> 1
    r_low = oracle.stable_rank_estimate(low, 20)
    assert 1.0 <= r_low < 1.01
    assert oracle.adaptive_uses_muon(low, 0.05, 20)                # 1 <= 0.05 * 30
    assert not oracle.adaptive_uses_muon(high, 0.05, 20)
    assert oracle.adaptive_uses_muon(low, r_low / 30, 20)          # equality takes Muon
    W = [rng.standard_normal((m, n)) * 0.02 for _ in range(3)] + [rng.standard_normal((1, 9))]
    G = [rng.standard_normal(w.shape) * 1e-2 for w in W]
    Ms = [low, high, low, rng.standard_normal((1, 9))]
    w, mm, d = oracle.lionmuon_adaptive_step(W, G, Ms, 3, 0.9, 0.99, 0.02, 0.01, 0.1, 0.05, 20,
                                             lion_only=[False, False, True, False])
    assert d == [True, False, False, False]
    ref_muon = oracle.lionmuon_update(W[0], G[0], Ms[0], 0, 1, 0.9, 0.99, 0.02, 0.01, 0.1)
    ref_lion = oracle.lionmuon_update(W[1], G[1], Ms[1], 1, 0, 0.9, 0.99, 0.02, 0.01, 0.1)
    assert np.array_equal(w[0], ref_muon[0]) and np.array_equal(w[1], ref_lion[0])

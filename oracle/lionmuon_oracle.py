"""Plain fp64 CPU oracle of the LionMuon optimizer step.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The GPU product
path (``paper_2605_19811_amd``) never imports it and shares no code, header,
constant table or helper with it.

Every function follows the paper (arXiv 2605.19811, "LionMuon: Alternating
Spectral and Sign Descent for Efficient Training"):

* Algorithm 1 (Section 3, "LionMuon and SignMuon"): the per-matrix update
  rule -- Lion interpolation, the ``t mod P`` branch between a Muon step and a
  Lion step, decoupled weight decay on both branches, and the momentum update
  done after the branch, every step.
* Section 2 (Related works, "Spectral methods" and "Approximating the matrix
  sign"): the Muon direction is msign(X) = U V^T approximated by K steps of an
  odd-polynomial Newton-Schulz iteration.
* Section 3, "Implementation notes": one momentum buffer per parameter; 1-D
  parameters do not take the spectral branch.
* Table 3 (Appendix D, full experimental configuration): K_NS = 5 and the optional NS
  output scaling 0.2*sqrt(max(m, n)).

Readings where the paper is silent:

* The quintic coefficients (a, b, c) = (3.4445, -4.7750, 2.0315) are the ones
  published with Muon (the paper cites it as the source of the NS step); the
  paper prints none.
* Frobenius pre-normalisation X0 = Ghat / (||Ghat||_F + eps), eps = 1e-7.
* A tall matrix (m > n) is iterated in transposed form; in exact arithmetic
  NS(X^T) = NS(X)^T, so this changes cost, not the result.
* sign(0) = 0.

All arithmetic is float64 numpy: a plain, obviously-correct restatement with
no blocking, no symmetry tricks and no batching. Pinned by
``tests/test_oracle.py`` against SVD closed forms, the textbook cubic
iteration's limit (the polar factor), brute force on tiny inputs and the
invariants the paper states.
"""
from __future__ import annotations

import math

import numpy as np

# Odd quintic p(x) = a*x + b*x^3 + c*x^5 of the Muon Newton-Schulz step
# (coefficients published with Muon; reading, the paper prints none).
QUINTIC = (3.4445, -4.7750, 2.0315)
# Classical cubic Newton-Schulz p(x) = 1.5*x - 0.5*x^3 (converges to U V^T).
CUBIC = (1.5, -0.5, 0.0)

NS_STEPS = 5          # K_NS, Table 3
NS_EPS = 1e-7         # Frobenius pre-normalisation guard (reading)

SCALE_NONE = 0        # Algorithm 1 uses NS output as is
SCALE_RMS02 = 1       # Table 3: NS output times 0.2*sqrt(max(m, n))


def is_muon_step(t: int, P: int) -> bool:
    """Branch rule of Algorithm 1: the Muon branch is taken iff t mod P == 0.

    P = 0 encodes P = infinity (the Muon branch is never taken).
    """
    if P < 0 or t < 0:
        raise ValueError("t and P must be non-negative")
    if P == 0:
        return False
    return t % P == 0


def elementwise_sign(x: np.ndarray) -> np.ndarray:
    """sign(x) with sign(0) = 0: the LMO of the max-norm (Section 2, notation)."""
    return np.sign(np.asarray(x, dtype=np.float64))


def ns_output_scale(m: int, n: int, scale_mode: int) -> float:
    """Optional NS output scaling of Table 3 (0.2*sqrt(max(m, n)))."""
    if scale_mode == SCALE_NONE:
        return 1.0
    if scale_mode == SCALE_RMS02:
        return 0.2 * math.sqrt(max(m, n))
    raise ValueError(f"unknown scale mode {scale_mode}")


def coefficient_schedule(steps: int, coeffs) -> list:
    """Per-step (a, b, c) list: one triple repeated ``steps`` times, or an
    explicit list of ``steps`` triples (an odd-polynomial schedule of the
    kind Section 2 mentions: classical, Polar Express, Chebyshev-type)."""
    c0 = np.asarray(coeffs, dtype=np.float64)
    if c0.ndim == 1:
        if c0.shape != (3,):
            raise ValueError("coefficients must be (a, b, c)")
        return [tuple(c0)] * steps
    if c0.shape != (steps, 3):
        raise ValueError("a schedule needs one (a, b, c) triple per step")
    return [tuple(r) for r in c0]


def newton_schulz(G: np.ndarray, steps: int = NS_STEPS, coeffs=QUINTIC,
                  eps: float = NS_EPS) -> np.ndarray:
    """NS_K(G): K Newton-Schulz steps towards msign(G) = U V^T (Section 2).

    X0 = G / (||G||_F + eps), oriented so that X has no more rows than
    columns; step k forms A = X X^T, B = b_k*A + c_k*A A and
    X <- a_k*X + B X; the result is turned back to G's orientation.
    ``coeffs`` is one (a, b, c) for every step or a list of per-step triples.
    """
    schedule = coefficient_schedule(steps, coeffs)
    X = np.array(G, dtype=np.float64, copy=True)
    if X.ndim != 2:
        raise ValueError("Newton-Schulz needs a 2-D matrix")
    transposed = X.shape[0] > X.shape[1]
    if transposed:
        X = X.T
    X = X / (np.linalg.norm(X, "fro") + eps)
    for a, b, c in schedule:
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    if transposed:
        X = X.T
    return X


def adamw_update(W, G, m, v, step, lr, beta1, beta2, eps, wd):
    """AdamW with decoupled weight decay (Loshchilov & Hutter), the fallback
    Section 3 names for 1-D parameters (Table 3: betas (0.8, 0.999), lr 1e-3):

        m <- beta1 m + (1-beta1) g;   v <- beta2 v + (1-beta2) g^2
        mhat = m / (1 - beta1^step);  vhat = v / (1 - beta2^step)
        W <- W - lr (mhat / (sqrt(vhat) + eps) + wd W)

    ``step`` counts AdamW steps from 1. Returns (W', m', v') in float64.
    """
    W, G, m, v = (np.asarray(x, dtype=np.float64) for x in (W, G, m, v))
    if step < 1:
        raise ValueError("AdamW steps count from 1")
    m_new = beta1 * m + (1.0 - beta1) * G
    v_new = beta2 * v + (1.0 - beta2) * G * G
    mhat = m_new / (1.0 - beta1 ** step)
    vhat = v_new / (1.0 - beta2 ** step)
    W_new = W - lr * (mhat / (np.sqrt(vhat) + eps) + wd * W)
    return W_new, m_new, v_new


def lionmuon_update(W, G, M, t, P, beta1, beta2, lr_muon, lr_lion, wd, *,
                    lion_only=False, ns_steps=NS_STEPS, coeffs=QUINTIC,
                    eps=NS_EPS, scale_mode=SCALE_NONE):
    """One step of Algorithm 1 for one parameter tensor, in float64.

    Ghat = beta1*M + (1-beta1)*G (interpolation with the PRE-update buffer);
    Muon branch (t mod P == 0, 2-D, not lion_only):
        W' = W - lr_muon * (kappa*NS_K(Ghat) + wd*W)
    Lion branch otherwise:
        W' = W - lr_lion * (sign(Ghat) + wd*W)
    then M' = beta2*M + (1-beta2)*G.  Returns (W', M').
    """
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    if not (W.shape == G.shape == M.shape):
        raise ValueError("W, G, M must have one shape")
    Ghat = beta1 * M + (1.0 - beta1) * G
    spectral = (W.ndim == 2 and min(W.shape) > 1 and not lion_only
                and is_muon_step(t, P))
    if spectral:
        kappa = ns_output_scale(W.shape[0], W.shape[1], scale_mode)
        direction = kappa * newton_schulz(Ghat, ns_steps, coeffs, eps)
        W_new = W - lr_muon * (direction + wd * W)
    else:
        W_new = W - lr_lion * (elementwise_sign(Ghat) + wd * W)
    M_new = beta2 * M + (1.0 - beta2) * G
    return W_new, M_new


def lionmuon_step(params, grads, moms, t, P, beta1, beta2, lr_muon, lr_lion,
                  wd, *, lion_only=None, **ns_kwargs):
    """Algorithm 1 applied to every tensor of a parameter list.

    ``lion_only`` is an optional per-tensor flag list; 1-D tensors never take
    the spectral branch (Section 3, implementation notes). Returns the lists
    (W', M') in float64.
    """
    n = len(params)
    if lion_only is None:
        lion_only = [False] * n
    out_w, out_m = [], []
    for W, G, M, lo in zip(params, grads, moms, lion_only):
        w, m = lionmuon_update(W, G, M, t, P, beta1, beta2, lr_muon, lr_lion,
                               wd, lion_only=lo, **ns_kwargs)
        out_w.append(w)
        out_m.append(m)
    return out_w, out_m


def stable_rank_estimate(M: np.ndarray, power_steps: int = 10,
                         v0: np.ndarray | None = None) -> float:
    """r_hat(M) = ||M||_F^2 / sigma_hat_1(M)^2 (Appendix G, adaptive rule).

    sigma_hat_1 comes from ``power_steps`` power-iteration steps on the Gram
    matrix of the short side: with S = M when M is tall or square and
    S = M^T when it is wide, v <- S^T S v / ||S^T S v|| from ``v0`` (length
    min(m, n), all-ones when not given, scaled to unit norm), and then
    sigma_hat_1 = ||S v||. The estimate is 0 when M = 0 or when an iterate
    vanishes.
    """
    M = np.asarray(M, dtype=np.float64)
    S = M.T if M.shape[0] < M.shape[1] else M
    s = S.shape[1]
    v = np.ones(s) if v0 is None else np.asarray(v0, dtype=np.float64)
    v = v / np.linalg.norm(v)
    for _ in range(power_steps):
        w = S.T @ (S @ v)
        nw = np.linalg.norm(w)
        if nw == 0.0:
            return 0.0
        v = w / nw
    sigma1 = np.linalg.norm(S @ v)
    if sigma1 == 0.0:
        return 0.0
    return float(np.linalg.norm(M, "fro") ** 2 / sigma1 ** 2)


def adaptive_uses_muon(M: np.ndarray, alpha: float, power_steps: int) -> bool:
    """Appendix G rule: the Muon step is taken on a matrix iff the stable rank
    of its momentum, r_hat(M) = ||M||_F^2 / sigma_hat_1^2, is at most
    alpha * min(m, n). M is the buffer before this step's update."""
    M = np.asarray(M, dtype=np.float64)
    return stable_rank_estimate(M, power_steps) <= alpha * min(M.shape)


def lionmuon_adaptive_step(params, grads, moms, t, beta1, beta2, lr_muon, lr_lion, wd, alpha,
                           power_steps, *, lion_only=None, **ns_kwargs):
    """One step of the adaptive variant (Appendix G): each 2-D matrix that is
    not Lion-only takes the Muon branch iff ``adaptive_uses_muon`` holds for
    its current momentum, the Lion branch otherwise; 1-D and Lion-only
    tensors take the Lion branch. Returns (W' list, M' list, decisions)."""
    n = len(params)
    lion_only = list(lion_only) if lion_only is not None else [False] * n
    out_w, out_m, decisions = [], [], []
    for W, G, M, lo in zip(params, grads, moms, lion_only):
        M64 = np.asarray(M, dtype=np.float64)
        eligible = M64.ndim == 2 and min(M64.shape) > 1 and not lo
        muon = eligible and adaptive_uses_muon(M64, alpha, power_steps)
        # P = 1 forces the Muon branch, P = 0 (infinity) the Lion branch
        w, m = lionmuon_update(W, G, M, t, 1 if muon else 0, beta1, beta2, lr_muon, lr_lion, wd,
                               lion_only=not muon, **ns_kwargs)
        out_w.append(w)
        out_m.append(m)
        decisions.append(bool(muon))
    return out_w, out_m, decisions

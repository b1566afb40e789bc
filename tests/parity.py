"""Comparison rules between the GPU step and the fp64 oracle.

Lion branch: the sign pattern must match exactly wherever the fp64 direction
is clear of the fp32 rounding band |Ghat| <= 2^-22 (beta1 |M| + (1-beta1)|G|);
inside the band (where fp32 rounding may give either sign or zero) the sign
must be one of -1, 0, +1 and W the admissible value for it, and the band
count is bounded. Weights and momentum within 1e-6 norm-wise relative error
(max-norm and Frobenius) of that reference.
Muon branch: the update direction recovered from W, (W - W')/eta_M - wd W,
within a relative Frobenius error of 2e-2 (bf16 MFMA path) or 1e-4 (fp32
path) of kappa NS_5(Ghat); momentum as on the Lion branch.
"""
import numpy as np

import oracle

LION_TOL = 1e-6
NS_TOL = {"bf16": 2e-2, "fp32": 1e-4}


def rel_max(a, b):
    den = np.abs(b).max()
    return float(np.abs(a - b).max() / den) if den > 0 else float(np.abs(a).max())


def rel_fro(a, b):
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a))


def check_momentum(M0, G, M_gpu, beta2):
    ref = beta2 * M0.astype(np.float64) + (1.0 - beta2) * G.astype(np.float64)
    assert rel_max(M_gpu, ref) <= LION_TOL, rel_max(M_gpu, ref)
    assert rel_fro(M_gpu, ref) <= LION_TOL, rel_fro(M_gpu, ref)


def band_limit(numel):
    """Largest rounding-band count a Lion-branch tensor of ``numel`` elements
    may show. With M and G independent and of one scale, the band holds with
    probability ~1.5e-7 per element (its width is 2^-22 of the terms); the
    limit leaves a wide margin over that rate plus a small constant for tiny
    tensors, so a kernel that spreads wrong signs over many elements fails."""
    return 4 + int(1e-6 * numel)


def check_lion(W0, G, M0, W_gpu, M_gpu, beta1, beta2, lr, wd, lion_only=True, max_band=None):
    """Lion branch against the oracle. Returns the number of rounding-band
    positions.

    Outside the band the sign of the update must equal the oracle's and W must
    match it. At a band position (``|Ghat| <= 2^-22 (beta1 |M| + (1-beta1) |G|)``,
    Ghat != 0) the fp32 interpolation may round to either sign or to zero, so
    the admissible results are ``W0 - lr (s + wd W0)`` with s in {-1, 0, +1}:
    the sign recovered from W must be one of those three and W must equal the
    admissible value for it. The band count is bounded by ``max_band``
    (default ``band_limit(W0.size)``); at M = 0 the band is empty (Ghat is
    exactly (1-beta1) G)."""
    W0d, Gd, M0d = (np.asarray(x, np.float64) for x in (W0, G, M0))
    w_ref, m_ref = oracle.lionmuon_update(W0d, Gd, M0d, 1, 0, beta1, beta2, 0.0, lr, wd,
                                          lion_only=lion_only)
    ghat = beta1 * M0d + (1.0 - beta1) * Gd
    band = np.abs(ghat) <= 2.0 ** -22 * (beta1 * np.abs(M0d) + (1.0 - beta1) * np.abs(Gd))
    band &= ghat != 0.0
    n_band = int(band.sum())
    limit = band_limit(W0d.size) if max_band is None else max_band
    assert n_band <= limit, f"{n_band} rounding-band positions (limit {limit})"
    if not M0d.any():
        assert n_band == 0, "rounding band must be empty when M = 0"
    W_gpu = np.asarray(W_gpu, np.float64)
    w_exp = w_ref.copy()
    if lr > 0:
        s_gpu = np.rint((W0d - W_gpu) / lr - wd * W0d)
        s_ref = np.sign(ghat)
        mism = (s_gpu != s_ref) & ~band
        assert not mism.any(), f"{int(mism.sum())} sign mismatches outside the rounding band"
        s_band = s_gpu[band]
        assert np.isin(s_band, (-1.0, 0.0, 1.0)).all(), \
            f"band positions hold signs {sorted(set(s_band.tolist()))}, not in {{-1, 0, +1}}"
        w_exp[band] = W0d[band] - lr * (s_band + wd * W0d[band])
    assert rel_max(W_gpu, w_exp) <= LION_TOL, rel_max(W_gpu, w_exp)
    assert rel_fro(W_gpu, w_exp) <= LION_TOL, rel_fro(W_gpu, w_exp)
    check_momentum(M0, G, M_gpu, beta2)
    return n_band


def muon_direction_error(W0, G, M0, W_gpu, beta1, lr, wd, kappa=1.0, steps=oracle.NS_STEPS):
    W0d = np.asarray(W0, np.float64)
    ghat = beta1 * np.asarray(M0, np.float64) + (1.0 - beta1) * np.asarray(G, np.float64)
    o_ref = kappa * oracle.newton_schulz(ghat, steps)
    o_gpu = (W0d - np.asarray(W_gpu, np.float64)) / lr - wd * W0d
    return rel_fro(o_gpu, o_ref)


def check_muon(W0, G, M0, W_gpu, M_gpu, beta1, beta2, lr, wd, precision, kappa=1.0,
               steps=oracle.NS_STEPS):
    err = muon_direction_error(W0, G, M0, W_gpu, beta1, lr, wd, kappa, steps)
    assert err <= NS_TOL[precision], f"Muon direction error {err:.3e} > {NS_TOL[precision]}"
    check_momentum(M0, G, M_gpu, beta2)
    return err


def check_adamw(W0, G, m0, v0, W_gpu, m_gpu, v_gpu, step, cfg):
    """AdamW tensors: weights and both moments within 1e-6 (max-norm and
    Frobenius relative) of the fp64 oracle."""
    w_ref, m_ref, v_ref = oracle.adamw_update(W0, G, m0, v0, step, cfg.adam_lr, cfg.adam_beta1,
                                              cfg.adam_beta2, cfg.adam_eps, cfg.adam_wd)
    for got, ref in ((W_gpu, w_ref), (m_gpu, m_ref), (v_gpu, v_ref)):
        got = np.asarray(got, np.float64)
        assert rel_max(got, ref) <= LION_TOL, rel_max(got, ref)
        assert rel_fro(got, ref) <= LION_TOL, rel_fro(got, ref)

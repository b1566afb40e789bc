"""CPU checks of the Lion-branch comparison rule in ``parity.check_lion``.

The GPU output is stood in for by an fp32 numpy evaluation of the Lion update
(test code, not the oracle). Inputs are built so that the interpolation
Ghat = beta1 M + (1-beta1) G cancels to within the fp32 rounding band at
chosen positions; there any of the signs -1, 0, +1 is an admissible result
(Algorithm 1's sign step applied to an fp32-rounded Ghat), and anything else
must fail the check.
"""
import numpy as np
import pytest

from parity import band_limit, check_lion

B1, B2, LR, WD = 0.9, 0.99, 1e-2, 0.1


def fp32_lion(W0, G, M0):
    """Lion step in fp32 arithmetic: the result a correct fp32 kernel may give."""
    f = np.float32
    c = f(B1) * M0 + f(1.0 - B1) * G
    W = W0 - f(LR) * (np.sign(c).astype(np.float32) + f(WD) * W0)
    M = f(B2) * M0 + f(1.0 - B2) * G
    return W.astype(np.float32), M.astype(np.float32)


def band_inputs(n=4096, n_band=3, seed=0):
    rng = np.random.default_rng(seed)
    W0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    M0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    G = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    # G = -beta1 M / (1 - beta1), rounded to fp32: Ghat is then a rounding
    # residue of the order 2^-24 of the terms, inside the band
    idx = np.arange(n_band) * 7 + 5
    G[idx] = (-B1 * M0[idx].astype(np.float64) / (1.0 - B1)).astype(np.float32)
    return W0, G, M0, idx


def band_mask(W0, G, M0):
    Md, Gd = M0.astype(np.float64), G.astype(np.float64)
    gh = B1 * Md + (1.0 - B1) * Gd
    return (np.abs(gh) <= 2.0 ** -22 * (B1 * np.abs(Md) + (1.0 - B1) * np.abs(Gd))) & (gh != 0)


def test_fp32_evaluation_passes_and_band_is_counted():
    W0, G, M0, idx = band_inputs()
    band = band_mask(W0, G, M0)
    assert band[idx].sum() >= 2, "construction puts positions in the band"
    W, M = fp32_lion(W0, G, M0)
    assert check_lion(W0, G, M0, W, M, B1, B2, LR, WD) == int(band.sum())


@pytest.mark.parametrize("s", [-1.0, 0.0, 1.0])
def test_every_admissible_band_value_passes(s):
    W0, G, M0, _ = band_inputs()
    band = band_mask(W0, G, M0)
    W, M = fp32_lion(W0, G, M0)
    W = W.astype(np.float64)
    W[band] = W0[band] - LR * (s + WD * W0[band].astype(np.float64))
    check_lion(W0, G, M0, W.astype(np.float32), M, B1, B2, LR, WD)


@pytest.mark.parametrize("bad", ["two", "untouched", "no_decay", "garbage"])
def test_wrong_value_at_a_band_position_fails(bad):
    W0, G, M0, _ = band_inputs()
    band = band_mask(W0, G, M0)
    pos = np.flatnonzero(band)[0]
    W, M = fp32_lion(W0, G, M0)
    W = W.astype(np.float64)
    w0 = float(W0[pos])
    W[pos] = {"two": w0 - LR * (2.0 + WD * w0),        # a sign of magnitude 2
              "untouched": w0,                          # no update written
              "no_decay": w0 - LR * 1.0,                # weight decay dropped
              "garbage": 0.5}[bad]
    with pytest.raises(AssertionError):
        check_lion(W0, G, M0, W.astype(np.float32), M, B1, B2, LR, WD)


def test_sign_flip_outside_the_band_fails():
    W0, G, M0, _ = band_inputs()
    band = band_mask(W0, G, M0)
    pos = np.flatnonzero(~band)[3]
    W, M = fp32_lion(W0, G, M0)
    W = W.astype(np.float64)
    s = np.sign(B1 * float(M0[pos]) + (1.0 - B1) * float(G[pos]))
    W[pos] = W0[pos] - LR * (-s + WD * float(W0[pos]))
    with pytest.raises(AssertionError):
        check_lion(W0, G, M0, W.astype(np.float32), M, B1, B2, LR, WD)


def test_too_many_band_positions_fail():
    n = 4096
    W0, G, M0, _ = band_inputs(n=n, n_band=band_limit(n) + 3)
    assert band_mask(W0, G, M0).sum() > band_limit(n)
    W, M = fp32_lion(W0, G, M0)
    with pytest.raises(AssertionError, match="rounding-band positions"):
        check_lion(W0, G, M0, W, M, B1, B2, LR, WD)


def test_band_is_empty_at_zero_momentum():
    rng = np.random.default_rng(3)
    W0 = (rng.standard_normal(10000) * 0.02).astype(np.float32)
    G = (rng.standard_normal(10000) * 1e-2).astype(np.float32)
    M0 = np.zeros_like(G)
    W, M = fp32_lion(W0, G, M0)
    assert check_lion(W0, G, M0, W, M, B1, B2, LR, WD) == 0


def test_band_rate_on_gaussian_state_is_far_below_the_limit():
    """The expected rate (~1.5e-7 per element for M, G of one scale): over 4M
    elements the count stays well under the limit."""
    rng = np.random.default_rng(4)
    n = 1 << 22
    M0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    G = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    W0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    count = int(band_mask(W0, G, M0).sum())
    assert count <= band_limit(n) // 2, count

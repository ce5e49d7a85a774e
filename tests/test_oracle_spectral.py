"""Pins of the oracle's spectral-decay analysis (Sec. 3.2; supplementary
Sec. S2): orthonormal 2-D DCT-II, radial bands, Pearson correlations by
lag, decorrelation horizons and the power-law fit.

The DCT is pinned to its definition (the cosine basis written out here,
orthonormal, applied as matrix products, and as explicit double sums on a
tiny frame) and to Parseval; Pearson to its identities; the band
correlations to exact cases (lag 0, repeated and negated frames) and to a
synthetic process with known per-band correlations; the fit to exact
power-law points.  The band partition, smoothing and horizon rule are
readings (the paper does not state them); parity unpinned as to the paper
for those.
"""
import math

import numpy as np
import pytest

from oracle import (band_correlations, dct2_ortho, decorrelation_horizons, fit_power_law, pearson,
                    radial_band_of)


def basis(N):
    n = np.arange(N)
    A = np.cos(np.pi * (2 * n[None, :] + 1) * n[:, None] / (2 * N))
    A[0] *= math.sqrt(1.0 / N)
    A[1:] *= math.sqrt(2.0 / N)
    return A


@pytest.mark.parametrize("H,W", [(6, 10), (60, 104), (7, 5)])
def test_dct_matches_the_cosine_basis(H, W):
    AH, AW = basis(H), basis(W)
    np.testing.assert_allclose(AH @ AH.T, np.eye(H), atol=1e-12)
    Z = np.random.default_rng(H).standard_normal((3, H, W))
    D = dct2_ortho(Z)
    np.testing.assert_allclose(D, AH @ Z @ AW.T, atol=1e-10)
    np.testing.assert_allclose((D ** 2).sum(axis=(1, 2)), (Z ** 2).sum(axis=(1, 2)), rtol=1e-12)  # Parseval


def test_dct_brute_force_and_single_basis_pattern():
    H, W = 3, 5
    Z = np.random.default_rng(1).standard_normal((H, W))
    D = dct2_ortho(Z)
    for u in range(H):
        for v in range(W):
            su = math.sqrt((1 if u == 0 else 2) / H)
            sv = math.sqrt((1 if v == 0 else 2) / W)
            ref = su * sv * sum(Z[h, w] * math.cos(math.pi * (2 * h + 1) * u / (2 * H)) *
                                math.cos(math.pi * (2 * w + 1) * v / (2 * W)) for h in range(H) for w in range(W))
            assert abs(D[u, v] - ref) < 1e-12
    P = np.outer(basis(8)[3], basis(12)[5])
    Dp = dct2_ortho(P)
    expect = np.zeros((8, 12))
    expect[3, 5] = 1.0
    np.testing.assert_allclose(Dp, expect, atol=1e-12)


def test_pearson_identities():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(200)
    y = rng.standard_normal(200)
    assert abs(pearson(x, x) - 1.0) < 1e-14
    assert abs(pearson(x, -x) + 1.0) < 1e-14
    assert abs(pearson(x, 3 * x + 7) - 1.0) < 1e-14
    assert abs(pearson(x, y) - pearson(2 * x - 1, 0.5 * y + 4)) < 1e-13
    assert abs(pearson(x, y) - np.corrcoef(x, y)[0, 1]) < 1e-13


def test_radial_bands():
    H, W, K = 60, 104, 24
    band, centres = radial_band_of(H, W, K)
    assert band.dtype == np.int32 and band.shape == (H, W) and band[0, 0] == -1
    rest = band.copy()
    rest[0, 0] = 0
    assert rest.min() >= 0 and rest.max() == K - 1
    r = np.sqrt((np.arange(H)[:, None] / H) ** 2 + (np.arange(W)[None, :] / W) ** 2)
    order = np.argsort(r, axis=None)
    flat = band.reshape(-1)[order][1:]
    assert np.all(np.diff(flat) >= 0)                   # bands follow r
    assert all((band == k).sum() >= 2 for k in range(K))  # every band holds a vector
    assert np.all(np.diff(centres) > 0)


def test_band_correlations_exact_cases():
    H, W, K, T = 12, 16, 6, 5
    band, _ = radial_band_of(H, W, K)
    rng = np.random.default_rng(3)
    z0 = rng.standard_normal((H, W))
    same = np.broadcast_to(z0, (1, T, H, W))
    np.testing.assert_allclose(band_correlations(same, band, K, T - 1), 1.0, atol=1e-12)
    flip = np.stack([z0 if t % 2 == 0 else -z0 for t in range(T)])[None]
    C = band_correlations(flip, band, K, T - 1)
    np.testing.assert_allclose(C[:, 1::2], -1.0, atol=1e-12)
    np.testing.assert_allclose(C[:, 0], 1.0, atol=1e-12)


def test_band_correlations_recover_known_per_band_decay():
    """DCT coefficients drawn as AR(1) processes with a known coefficient per
    band: C_k(lag) must come out near rho_k^lag."""
    H, W, K, T, clips = 24, 32, 4, 6, 12
    band, _ = radial_band_of(H, W, K)
    rho = np.array([0.95, 0.8, 0.6, 0.3])
    AH, AW = basis(H), basis(W)
    rng = np.random.default_rng(4)
    lat = np.zeros((clips, T, H, W))
    r = np.where(band >= 0, rho[np.maximum(band, 0)], 0.0)
    for c in range(clips):
        d = rng.standard_normal((H, W))
        for t in range(T):
            if t:
                d = r * d + np.sqrt(1 - r ** 2) * rng.standard_normal((H, W))
            lat[c, t] = AH.T @ d @ AW
    C = band_correlations(lat, band, K, T - 1)
    expect = rho[:, None] ** np.arange(T)[None, :]
    np.testing.assert_allclose(C, expect, atol=0.06)


def test_horizons_and_power_law_fit():
    lags = np.arange(200)
    taus = np.array([40.0, 20.0, 10.0, 5.0])
    curves = np.exp(-lags[None, :] / taus[:, None]) * 0.9 + 0.1
    h = decorrelation_horizons(curves)
    assert np.all(h > 0) and np.all(np.diff(h) < 0)               # slower decay, later horizon
    np.testing.assert_allclose(h / taus, math.log(20.0), rtol=0.15)  # about tau * ln 20 for exp(-lag/tau)
    t = np.array([2.0, 3.0, 5.0, 8.0, 13.0, 21.0])
    a, b = fit_power_law(t, 0.7 * t ** -0.45)
    assert abs(a - 0.7) < 1e-8 and abs(b - 0.45) < 1e-8

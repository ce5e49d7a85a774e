"""The library's host steps of the spectral-decay analysis (Sec. 3.2;
supplementary Sec. S2) against the oracle: the radial band map, the
decorrelation horizons and the power-law fit.  They run on the host and
need no GPU."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2606_10671_amd import fademem as fm
from paper_2606_10671_amd import spectral as sp


@pytest.mark.parametrize("H,W,bands", [(60, 104, 24), (1, 1, 1), (1, 7, 3), (9, 2, 5), (64, 128, 40),
                                       (33, 17, 1024), (1024, 3, 7)])
def test_band_map_equals_the_oracle(H, W, bands):
    got, centres = sp.radial_band_map(H, W, bands)
    ref, ref_centres = oracle.radial_band_of(H, W, bands)
    assert got.dtype == np.int32 and got.shape == (H, W)
    assert np.array_equal(got, ref)
    assert np.array_equal(centres, ref_centres)


def synthetic_curves(rng, bands, lags):
    t = np.arange(lags, dtype=np.float64)
    taus = rng.uniform(2.0, 40.0, size=bands)
    floor = rng.uniform(0.0, 0.3, size=bands)
    noise = rng.normal(0.0, 0.01, size=(bands, lags))
    return (1 - floor)[:, None] * np.exp(-t[None, :] / taus[:, None]) + floor[:, None] + noise


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("width,drop", [(5, 0.05), (1, 0.05), (3, 0.2), (9, 0.01)])
def test_horizons_equal_the_oracle(seed, width, drop):
    rng = np.random.default_rng(seed)
    curves = synthetic_curves(rng, 24, 177)
    got = sp.decorrelation_horizons(curves, width=width, drop=drop)
    assert np.array_equal(got, oracle.decorrelation_horizons(curves, width=width, drop=drop))


def test_horizon_edge_cases():
    flat = np.ones((1, 20))
    rising = np.linspace(0.0, 1.0, 20)[None, :]
    short = np.array([[1.0, 0.5]])
    single = np.array([[1.0]])
    nan = np.full((1, 10), np.nan)
    for c in (flat, rising, short, single, nan):
        assert np.array_equal(sp.decorrelation_horizons(c), oracle.decorrelation_horizons(c)), c
        assert sp.decorrelation_horizons(c)[0] == -1


@pytest.mark.parametrize("a,b,n,noise", [(0.7, 0.45, 12, 0.0), (0.3, 0.2, 6, 0.02), (2.0, 1.1, 30, 0.01),
                                         (0.5, -0.3, 5, 0.0)])
def test_fit_matches_the_oracle(a, b, n, noise):
    rng = np.random.default_rng(3)
    t = np.sort(rng.uniform(1.0, 120.0, size=n))
    r = a * t ** (-b) * (1.0 + noise * rng.standard_normal(n))
    ga, gb = sp.fit_power_law(t, r)
    oa, ob = oracle.fit_power_law(t, r)
    assert abs(ga - oa) <= 1e-6 * abs(oa) and abs(gb - ob) <= 1e-6 * max(abs(ob), 1e-3), (ga, gb, oa, ob)
    if noise == 0.0:
        assert abs(ga - a) <= 1e-9 * a and abs(gb - b) <= 1e-9 * max(abs(b), 1.0)


def test_host_step_errors():
    L = fm.lib()
    buf = (ctypes.c_int32 * 4)()
    assert L.fademem_spectral_band_map(0, 4, 2, buf, None) == fm.FADEMEM_EINVAL
    assert L.fademem_spectral_band_map(2, 2, 0, buf, None) == fm.FADEMEM_EINVAL
    assert L.fademem_spectral_band_map(2, 2, 2, None, None) == fm.FADEMEM_EINVAL
    h = (ctypes.c_int64 * 2)()
    c = (ctypes.c_double * 4)()
    assert L.fademem_spectral_horizons(None, 2, 2, 5, 0.05, h) == fm.FADEMEM_EINVAL
    assert L.fademem_spectral_horizons(c, 2, 2, 0, 0.05, h) == fm.FADEMEM_EINVAL
    t = np.array([1.0, 1.0, 1.0])
    with pytest.raises(fm.FademError):
        sp.fit_power_law(t, np.array([1.0, 2.0, 3.0]))        # the exponent is not determined
    with pytest.raises(fm.FademError):
        sp.fit_power_law(np.array([1.0, -2.0]), np.array([1.0, 2.0]))
    with pytest.raises(fm.FademError):
        sp.fit_power_law(np.array([1.0]), np.array([1.0]))

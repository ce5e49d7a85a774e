"""GPU parity of the spectral-decay analysis (Sec. 3.2; supplementary
Sec. S2): the library's DCT + band-correlation pipeline against the oracle
(fp64 DCT, Pearson by definition), within 1e-5 absolute on every C_k(lag)
(the kernels transform in fp32 and sum in fp64).  The host analysis of the
package (horizons, power-law fit) is compared with the oracle's on the same
curves.  Inputs: random frames, and synthetic multi-scale clips at the
paper's latent shape (60 x 104, 177 frames; the paper's videos and VAE are
not available)."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2606_10671_amd.synth import SpectralClips

pytestmark = pytest.mark.gpu

CORR_ABS = 1e-5


def gpu_corr(lat_np, band_np, bands, max_lag):
    import torch
    from paper_2606_10671_amd import spectral as sp
    lat = torch.from_numpy(np.ascontiguousarray(lat_np, dtype=np.float32)).cuda()
    band = torch.from_numpy(np.ascontiguousarray(band_np, dtype=np.int32)).cuda()
    return sp.spectral_corr(lat, band, bands, max_lag).cpu().numpy()


# Frames up to 64 x 128 take the fused matrix-core kernel (1 to 4 tiles of 16
# rows); larger ones the general two-kernel path.
@pytest.mark.parametrize("clips,frames,H,W,bands,max_lag", [
    (3, 12, 20, 36, 8, 11),      # fused, 2 row tiles, ragged columns
    (1, 5, 7, 9, 3, 2),          # fused, 1 row tile
    (2, 10, 40, 64, 12, 9),      # fused, 3 row tiles, full column tiles
    (4, 9, 60, 104, 24, 0),      # fused, the paper's latent shape, lag 0 only
    (5, 13, 64, 128, 16, 12),    # fused, largest shape
    (2, 6, 96, 100, 16, 5),      # general path (rows > 64)
    (2, 7, 40, 130, 10, 6),      # general path (columns > 128)
])
def test_spectral_parity_random(clips, frames, H, W, bands, max_lag):
    print(f"spectral clips={clips} frames={frames} H={H} W={W} bands={bands} max_lag={max_lag}", flush=True)
    lat = np.random.default_rng(H * W + frames).standard_normal((clips, frames, H, W)).astype(np.float32)
    band, _ = oracle.radial_band_of(H, W, bands)
    got = gpu_corr(lat, band, bands, max_lag)
    ref = oracle.band_correlations(lat, band, bands, max_lag)
    assert np.abs(got - ref).max() <= CORR_ABS, np.abs(got - ref).max()
    np.testing.assert_allclose(got[:, 0], 1.0, atol=1e-9)


@pytest.mark.parametrize("H,W,bands", [(64, 128, 1024), (60, 104, 300)])
def test_spectral_many_bands_with_empty_ones(H, W, bands):
    """Fine partitions leave bands with fewer than two coefficients: their
    coefficient is NaN on both sides; every other one within the bar."""
    print(f"spectral many bands H={H} W={W} bands={bands}", flush=True)
    lat = np.random.default_rng(bands).standard_normal((3, 5, H, W)).astype(np.float32)
    band, _ = oracle.radial_band_of(H, W, bands)
    got = gpu_corr(lat, band, bands, 4)
    with np.errstate(invalid="ignore", divide="ignore"):
        import warnings
        with warnings.catch_warnings():
            warnings.simplefilter("ignore")
            ref = oracle.band_correlations(lat, band, bands, 4)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert ok.sum() > 0
    assert np.abs(got[ok] - ref[ok]).max() <= CORR_ABS


def test_spectral_band_map_with_left_out_coefficients():
    H, W, bands, max_lag = 16, 24, 5, 4
    lat = np.random.default_rng(8).standard_normal((2, 6, H, W)).astype(np.float32)
    band, _ = oracle.radial_band_of(H, W, bands)
    band = band.copy()
    band[::3, ::2] = -1          # left out
    band[1, 1] = 77              # outside [0, bands): left out too
    ref_band = np.where((band >= 0) & (band < bands), band, -1)
    got = gpu_corr(lat, band, bands, max_lag)
    ref = oracle.band_correlations(lat, ref_band, bands, max_lag)
    assert np.abs(got - ref).max() <= CORR_ABS


def test_spectral_paper_shape_and_power_law():
    """Six synthetic clips of 177 latent frames at 60 x 104, 24 bands, every
    lag: parity, then horizons and the power-law fit of r*(t)."""
    from paper_2606_10671_amd import spectral as sp
    clips, T, H, W, bands = 6, 177, 60, 104, 24
    print(f"spectral paper shape clips={clips} T={T}", flush=True)
    gen = SpectralClips(5, T, H, W)
    lat = np.stack([gen.clip().numpy() for _ in range(clips)])
    band, centres = sp.radial_band_map(H, W, bands)
    got = gpu_corr(lat, band, bands, T - 1)
    ref = oracle.band_correlations(lat, band, bands, T - 1)
    assert np.abs(got - ref).max() <= CORR_ABS, np.abs(got - ref).max()
    h = sp.decorrelation_horizons(got)
    assert np.array_equal(h, oracle.decorrelation_horizons(got))
    ok = h > 0
    assert ok.sum() >= 4
    a, b = sp.fit_power_law(h[ok].astype(np.float64), centres[ok])
    ao, bo = oracle.fit_power_law(h[ok].astype(np.float64), centres[ok])
    assert abs(a - ao) <= 1e-6 * abs(ao) and abs(b - bo) <= 1e-6 * max(abs(bo), 1e-3)
    print(f"horizons {h.tolist()} fit a={a:.4f} b={b:.4f}", flush=True)
    assert b > 0  # the stable radius shrinks with distance on this data


def test_spectral_argument_errors():
    import torch
    from paper_2606_10671_amd import fademem as fm
    L = fm.lib()
    n = ctypes.c_size_t(0)
    assert L.fademem_spectral_workspace_bytes(2, 5, 8, 8, 4, 5, ctypes.byref(n)) == fm.FADEMEM_EINVAL  # lag >= frames
    assert L.fademem_spectral_workspace_bytes(2, 5, 300, 300, 4, 2, ctypes.byref(n)) == fm.FADEMEM_EINVAL  # LDS
    assert L.fademem_spectral_workspace_bytes(2, 5, 8, 8, 0, 2, ctypes.byref(n)) == fm.FADEMEM_EINVAL
    assert L.fademem_spectral_workspace_bytes(2, 5, 8, 8, 4, 2, ctypes.byref(n)) == fm.FADEMEM_OK
    need = n.value
    lat = torch.zeros((2, 5, 8, 8), dtype=torch.float32, device="cuda")
    band = torch.zeros((8, 8), dtype=torch.int32, device="cuda")
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    corr = torch.empty((4, 3), dtype=torch.float64, device="cuda")
    args = lambda wsb: (ctypes.c_void_p(lat.data_ptr()), 2, 5, 8, 8, ctypes.c_void_p(band.data_ptr()), 4, 2,
                        ctypes.c_void_p(ws.data_ptr()), wsb, ctypes.c_void_p(corr.data_ptr()), None)
    assert L.fademem_spectral_corr(*args(need - 1)) == fm.FADEMEM_ENOMEM
    assert L.fademem_spectral_corr(None, 2, 5, 8, 8, None, 4, 2, None, need, None, None) == fm.FADEMEM_EINVAL


def test_spectral_full_workload_and_determinism():
    """The benchmark's workload: 374 clips (32 distinct seeded clips, cycled)
    of 177 latent frames at 60 x 104, 24 bands, every lag.  The clip mean is
    linear, so the oracle's per-clip curves of the 32 distinct clips,
    weighted by how often each occurs, give the expected mean exactly; every
    C_k(lag) is checked.  Two calls give the same bits."""
    import torch
    from paper_2606_10671_amd import spectral as sp
    C, T, H, W, K, distinct = 374, 177, 60, 104, 24, 32
    print(f"spectral full workload clips={C} T={T} {H}x{W} bands={K}", flush=True)
    gen = SpectralClips(0, T, H, W)  # host generator (seconds), then one copy to the device
    clips = [gen.clip() for _ in range(distinct)]
    lat = torch.stack([clips[c % distinct] for c in range(C)]).cuda().contiguous()
    band_np, _ = sp.radial_band_map(H, W, K)
    band = torch.from_numpy(band_np).cuda()
    got = sp.spectral_corr(lat, band, K, T - 1).cpu().numpy()
    again = sp.spectral_corr(lat, band, K, T - 1).cpu().numpy()
    assert np.array_equal(got.view(np.uint64), again.view(np.uint64))
    counts = np.bincount(np.arange(C) % distinct, minlength=distinct)
    ref = np.zeros((K, T))
    for d in range(distinct):
        ref += counts[d] * oracle.band_correlations(clips[d].cpu().numpy()[None], band_np, K, T - 1)
    ref /= C
    assert np.abs(got - ref).max() <= CORR_ABS, np.abs(got - ref).max()


@pytest.mark.parametrize("clips,frames,H,W,bands,max_lag", [(3, 7, 60, 104, 40, 6), (2, 5, 70, 90, 12, 4)])
def test_spectral_arbitrary_band_map(clips, frames, H, W, bands, max_lag):
    """Bands need not be radial: a random assignment (some bands empty,
    some coefficients left out), on the fused (60 x 104) and the general
    (70 x 90) path."""
    print(f"spectral random bands {H}x{W} bands={bands}", flush=True)
    rng = np.random.default_rng(bands)
    lat = rng.standard_normal((clips, frames, H, W)).astype(np.float32)
    band = rng.integers(-1, bands - 3, (H, W)).astype(np.int32)  # the last three bands stay empty
    got = gpu_corr(lat, band, bands, max_lag)
    import warnings
    with np.errstate(invalid="ignore", divide="ignore"), warnings.catch_warnings():
        warnings.simplefilter("ignore")
        ref = oracle.band_correlations(lat, band, bands, max_lag)
    assert np.array_equal(np.isnan(got), np.isnan(ref)) and np.isnan(got[-3:]).all()
    ok = ~np.isnan(ref)
    assert np.abs(got[ok] - ref[ok]).max() <= CORR_ABS


@pytest.mark.parametrize("clips,frames,H,W,bands,max_lag", [(1, 1, 1, 1, 1, 0), (2, 1, 16, 16, 4, 0)])
def test_spectral_degenerate(clips, frames, H, W, bands, max_lag):
    """One frame (lag 0 only); a 1 x 1 frame whose single coefficient forms
    the only band: a band of one coefficient has no spread, so NaN."""
    lat = np.random.default_rng(H).standard_normal((clips, frames, H, W)).astype(np.float32)
    band = np.zeros((1, 1), np.int32) if H * W == 1 else oracle.radial_band_of(H, W, bands)[0]
    got = gpu_corr(lat, band, bands, max_lag)
    assert got.shape == (bands, 1)
    if H * W == 1:
        assert np.isnan(got).all()
    else:
        np.testing.assert_allclose(got, 1.0, atol=1e-9)

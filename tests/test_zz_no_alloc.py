"""The allocation-free spectral entry point (fademem_spectral_corr_static,
for callers that cannot allocate device memory) against the existing one
(fademem_spectral_corr with a caller's workspace), through the C ABI: two
calls in a row, the second with a smaller input, each bit for bit equal to
the workspace entry point's result (the same kernels), and within the
oracle's bar; an oversized request is refused before anything runs."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

CORR_ABS = 1e-5


def both(lat_np, bands, max_lag):
    import torch
    from paper_2606_10671_amd import fademem as fm
    from paper_2606_10671_amd import spectral as sp
    clips, frames, H, W = lat_np.shape
    band_np, _ = sp.radial_band_map(H, W, bands)
    lat = torch.from_numpy(np.ascontiguousarray(lat_np, dtype=np.float32)).cuda()
    band = torch.from_numpy(band_np).cuda()
    ref = sp.spectral_corr(lat, band, bands, max_lag)
    got = torch.full((bands, max_lag + 1), float("nan"), dtype=torch.float64, device="cuda")
    fm.fademem_spectral_corr_static(lat.data_ptr(), clips, frames, H, W, band.data_ptr(), bands, max_lag,
                                    got.data_ptr(), int(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    return got.cpu().numpy(), ref.cpu().numpy(), band_np


def test_static_scratch_matches_the_workspace_entry_point():
    rng = np.random.default_rng(4)
    print("no-alloc spectral: first call 6 clips x 40 frames of 60 x 104, 24 bands", flush=True)
    lat1 = rng.standard_normal((6, 40, 60, 104)).astype(np.float32)
    got1, ref1, band1 = both(lat1, 24, 39)
    assert np.array_equal(got1.view(np.uint64), ref1.view(np.uint64))
    assert np.abs(got1 - oracle.band_correlations(lat1, band1, 24, 39)).max() <= CORR_ABS
    print("no-alloc spectral: second call 2 clips x 9 frames of 20 x 36, 8 bands", flush=True)
    lat2 = rng.standard_normal((2, 9, 20, 36)).astype(np.float32)
    got2, ref2, band2 = both(lat2, 8, 8)
    assert np.array_equal(got2.view(np.uint64), ref2.view(np.uint64))
    assert np.abs(got2 - oracle.band_correlations(lat2, band2, 8, 8)).max() <= CORR_ABS


def test_static_scratch_refuses_oversized_requests():
    import torch
    from paper_2606_10671_amd import fademem as fm
    # 4000 clips x 200 lags x 24 bands of band sums: 461 MB, beyond the 64 MiB scratch
    need = fm.fademem_spectral_workspace_bytes(4000, 200, 60, 104, 24, 199)
    assert need > 64 << 20
    lat = torch.zeros(16, dtype=torch.float32, device="cuda")
    band = torch.zeros(16, dtype=torch.int32, device="cuda")
    corr = torch.zeros(16, dtype=torch.float64, device="cuda")
    with pytest.raises(fm.FademError) as e:
        fm.fademem_spectral_corr_static(lat.data_ptr(), 4000, 200, 60, 104, band.data_ptr(), 24, 199,
                                        corr.data_ptr(), 0)
    assert e.value.code == fm.FADEMEM_ESCRATCH
    assert int(torch.count_nonzero(corr)) == 0

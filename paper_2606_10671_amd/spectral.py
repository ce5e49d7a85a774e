"""Distance-dependent spectral decay (FadeMem Sec. 3.2; supplementary Sec. S2).

Argument marshalling for the library's spectral calls (include/fademem.h):

* ``spectral_corr`` -- the HIP pipeline: orthonormal 2-D DCT-II of every
  latent frame, Pearson correlation of each radial band's coefficients
  between frame 0 and frame lag, mean over clips;
* ``radial_band_map``, ``decorrelation_horizons``, ``fit_power_law`` -- the
  library's host steps on the result (band map, horizons, power-law fit).

The band partition, smoothing and horizon rule are readings: the paper
does not state them.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from . import fademem as fm


def radial_band_map(height: int, width: int, bands: int) -> Tuple[np.ndarray, np.ndarray]:
    """int32 [height][width] band index per DCT coefficient (-1 = left out)
    and float64 [bands] centre radii (fademem_spectral_band_map)."""
    band_of = np.empty((height, width), dtype=np.int32)
    centres = np.empty(bands, dtype=np.float64)
    fm.fademem_spectral_band_map(height, width, bands, band_of.ctypes.data, centres.ctypes.data)
    return band_of, centres


def spectral_corr(latents, band_of, bands: int, max_lag: int, stream=None):
    """C_k(lag), a float64 [bands][max_lag+1] CUDA tensor.  latents: float32
    CUDA tensor [clips][frames][H][W]; band_of: int32 CUDA tensor [H][W]."""
    import torch
    if latents.dtype != torch.float32 or latents.dim() != 4 or not latents.is_contiguous():
        raise ValueError("latents: expected a contiguous float32 [clips][frames][H][W] tensor")
    clips, frames, H, W = (int(x) for x in latents.shape)
    if band_of.dtype != torch.int32 or tuple(band_of.shape) != (H, W) or not band_of.is_contiguous():
        raise ValueError("band_of: expected a contiguous int32 [H][W] tensor")
    need = fm.fademem_spectral_workspace_bytes(clips, frames, H, W, bands, max_lag)
    ws = torch.empty(need, dtype=torch.uint8, device=latents.device)
    corr = torch.empty((bands, max_lag + 1), dtype=torch.float64, device=latents.device)
    s = torch.cuda.current_stream() if stream is None else stream
    fm.fademem_spectral_corr(latents.data_ptr(), clips, frames, H, W, band_of.data_ptr(), bands, max_lag,
                             ws.data_ptr(), need, corr.data_ptr(), int(s.cuda_stream))
    return corr


def decorrelation_horizons(corr, width: int = 5, drop: float = 0.05) -> np.ndarray:
    """int64 [bands] horizon lag per band, -1 where the curve never flattens
    (fademem_spectral_horizons)."""
    c = np.ascontiguousarray(corr, dtype=np.float64)
    out = np.empty(c.shape[0], dtype=np.int64)
    fm.fademem_spectral_horizons(c.ctypes.data, c.shape[0], c.shape[1], width, drop, out.ctypes.data)
    return out


def fit_power_law(t, r, iters: int = 100) -> Tuple[float, float]:
    """(a, b) minimising sum (r_i - a t_i^(-b))^2 (fademem_spectral_fit)."""
    t = np.ascontiguousarray(t, dtype=np.float64)
    r = np.ascontiguousarray(r, dtype=np.float64)
    if t.shape != r.shape or t.ndim != 1:
        raise ValueError("t and r: expected 1-D arrays of the same length")
    return fm.fademem_spectral_fit(t.ctypes.data, r.ctypes.data, len(t), iters)

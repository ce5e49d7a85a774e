"""Distance-dependent spectral decay (FadeMem Sec. 3.2; supplementary Sec. S2).

``spectral_corr`` runs the library's HIP pipeline (orthonormal 2-D DCT-II of
every latent frame, Pearson correlation of each radial band's coefficients
between frame 0 and frame lag, mean over clips).  The rest is a few dozen
numbers of host work on its result:

* ``radial_band_map`` -- `bands` equal-width bands of the normalized radial
  frequency r(u, v) = sqrt((u/H)^2 + (v/W)^2) over [0, max r], the DC
  coefficient left out, and the bands' centre radii;
* ``decorrelation_horizons`` -- per band, the smoothed curve (centred moving
  average over 5 lags, shrinking at the ends) enters its near-flat regime at
  the first lag, after at least half of its total decay, where it falls by
  less than 5 % of its steepest one-lag fall;
* ``fit_power_law`` -- r*(t) = a t^(-b) by nonlinear least squares
  (Gauss-Newton on the residuals, started from the log-log line).

The band partition, smoothing and horizon rule are readings: the paper
does not state them.
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np

from . import fademem as fm


def radial_band_map(height: int, width: int, bands: int) -> Tuple[np.ndarray, np.ndarray]:
    """int32 [height][width] band index per DCT coefficient (-1 = left out)
    and float64 [bands] centre radii."""
    u = np.arange(height, dtype=np.float64).reshape(-1, 1) / height
    v = np.arange(width, dtype=np.float64).reshape(1, -1) / width
    r = np.hypot(u, v)
    top = float(r.max())
    idx = np.floor(r * (bands / top)).astype(np.int64)
    idx = np.clip(idx, 0, bands - 1).astype(np.int32)
    idx[0, 0] = -1
    centres = (np.arange(bands, dtype=np.float64) + 0.5) * (top / bands)
    return idx, centres


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


def _smooth(curve: np.ndarray, width: int) -> np.ndarray:
    h = width // 2
    n = len(curve)
    c = np.concatenate([[0.0], np.cumsum(curve)])
    lo = np.maximum(np.arange(n) - h, 0)
    hi = np.minimum(np.arange(n) + h + 1, n)
    return (c[hi] - c[lo]) / (hi - lo)


def decorrelation_horizons(corr, width: int = 5, drop: float = 0.05) -> np.ndarray:
    """int64 [bands] horizon lag per band (-1 where the curve never flattens)."""
    corr = np.asarray(corr, dtype=np.float64)
    out = np.full(corr.shape[0], -1, dtype=np.int64)
    for k, curve in enumerate(corr):
        s = _smooth(curve, width)
        falls = s[:-1] - s[1:]
        total = s[0] - s.min()
        if len(falls) == 0 or not (total > 0 and falls.max() > 0):
            continue
        ok = (s[0] - s[:-1] >= 0.5 * total) & (falls < drop * falls.max())
        ok[0] = False
        hits = np.nonzero(ok)[0]
        if len(hits):
            out[k] = int(hits[0])
    return out


def fit_power_law(t, r, iters: int = 100) -> Tuple[float, float]:
    """(a, b) minimising sum (r_i - a t_i^(-b))^2 by Gauss-Newton."""
    t = np.asarray(t, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    lt = np.log(t)
    slope, icpt = np.polyfit(lt, np.log(r), 1)
    a, b = math.exp(icpt), -slope
    for _ in range(iters):
        f = a * np.exp(-b * lt)
        res = r - f
        J = np.stack([f / a, -lt * f], axis=1)  # d f / d(a, b)
        step, *_ = np.linalg.lstsq(J, res, rcond=None)
        a, b = a + step[0], b + step[1]
        if abs(step[0]) <= 1e-14 * max(1.0, abs(a)) and abs(step[1]) <= 1e-14 * max(1.0, abs(b)):
            break
    return float(a), float(b)

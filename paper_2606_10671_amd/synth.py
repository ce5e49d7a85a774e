"""Seeded synthetic inputs with the shapes of the paper's workload.

This module only draws random numbers; it holds none of FadeMem's
arithmetic, and both the tests' oracle side and the library side consume
what it produces.  (The paper's generator weights, prompts and videos are
not available, so synthetic K/V stand in for them.)

Recipes
-------
* tiny: per step, Q, K, V i.i.d. N(0, 1) fp32 of shape [64][2][64], drawn
  in the order Q, K, V from numpy's default_rng(seed).
* Wan-class streams: per frame f and element x,
      m_0 = z_0,   m_f = rho * m_{f-1} + sqrt(1 - rho^2) * z_f   (rho = 0.95)
      K_f = m_f + 0.5 * e_f
  with z, e i.i.d. N(0, 1); V likewise from independent draws; Q i.i.d.
  N(0, 1); all rounded to bf16.  A chunk's F frames are consecutive frames
  of the stream, so merged neighbours are correlated but not identical.
* spectral clips (``SpectralClips``): per frame, the sum of five random
  fields, field s being white noise box-filtered with half-width w_s and
  evolving over frames as AR(1) with coefficient rho_s, each scaled to unit
  standard deviation (coarse scales decorrelate slowly, fine ones fast).
"""
from __future__ import annotations

import numpy as np

RHO = 0.95
NOISE_STD = 0.5


def tiny_steps(seed: int = 0, steps: int = 40, tokens: int = 64, heads: int = 2, head_dim: int = 64):
    """Yield (Q, K, V) float32 arrays [tokens][heads][head_dim] per step."""
    rng = np.random.default_rng(seed)
    shape = (tokens, heads, head_dim)
    for _ in range(steps):
        q = rng.standard_normal(shape, dtype=np.float32)
        k = rng.standard_normal(shape, dtype=np.float32)
        v = rng.standard_normal(shape, dtype=np.float32)
        yield q, k, v


class NumpyWanStream:
    """Host (numpy) version of the AR(1) K/V stream, for small shapes.

    ``frame()`` returns float32 arrays of bf16 values (K, V) [N][H][D];
    ``queries(n)`` returns bf16-valued float32 Q [n][H][D]."""

    def __init__(self, seed: int, tokens: int, heads: int, head_dim: int, rho: float = RHO,
                 noise_std: float = NOISE_STD):
        self.rng = np.random.default_rng(seed)
        self.shape = (tokens, heads, head_dim)
        self.rho, self.noise_std = rho, noise_std
        self.mk = None
        self.mv = None

    @staticmethod
    def _bf16(x: np.ndarray) -> np.ndarray:
        import torch
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).float().numpy()

    def frame(self):
        z_k = self.rng.standard_normal(self.shape, dtype=np.float32)
        z_v = self.rng.standard_normal(self.shape, dtype=np.float32)
        if self.mk is None:
            self.mk, self.mv = z_k, z_v
        else:
            a = np.float32(self.rho)
            b = np.float32(np.sqrt(1.0 - self.rho ** 2))
            self.mk = a * self.mk + b * z_k
            self.mv = a * self.mv + b * z_v
        k = self.mk + np.float32(self.noise_std) * self.rng.standard_normal(self.shape, dtype=np.float32)
        v = self.mv + np.float32(self.noise_std) * self.rng.standard_normal(self.shape, dtype=np.float32)
        return self._bf16(k), self._bf16(v)

    def queries(self, n: int):
        q = self.rng.standard_normal((n,) + self.shape[1:], dtype=np.float32)
        return self._bf16(q)


class TorchWanStream:
    """Device (torch) version of the AR(1) stream for full-size shapes.

    ``chunk(F)`` returns (Q, K, V) bf16 CUDA tensors of [F*N][H][D]; the K, V
    rows of frame f are rows f*N .. (f+1)*N-1."""

    def __init__(self, seed: int, tokens: int, heads: int, head_dim: int, device="cuda", rho: float = RHO,
                 noise_std: float = NOISE_STD):
        import torch
        self.torch = torch
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed)
        self.shape = (tokens, heads, head_dim)
        self.device = device
        self.rho, self.noise_std = rho, noise_std
        self.mk = None
        self.mv = None

    def _randn(self, shape):
        return self.torch.randn(shape, generator=self.gen, device=self.device, dtype=self.torch.float32)

    def frame(self):
        z_k, z_v = self._randn(self.shape), self._randn(self.shape)
        if self.mk is None:
            self.mk, self.mv = z_k, z_v
        else:
            b = float(np.sqrt(1.0 - self.rho ** 2))
            self.mk = self.rho * self.mk + b * z_k
            self.mv = self.rho * self.mv + b * z_v
        k = self.mk + self.noise_std * self._randn(self.shape)
        v = self.mv + self.noise_std * self._randn(self.shape)
        return k.to(self.torch.bfloat16), v.to(self.torch.bfloat16)

    def chunk(self, frames: int):
        ks, vs = zip(*[self.frame() for _ in range(frames)])
        q = self._randn((frames * self.shape[0],) + self.shape[1:]).to(self.torch.bfloat16)
        return q, self.torch.cat(ks, 0).contiguous(), self.torch.cat(vs, 0).contiguous()


class SpectralClips:
    """Synthetic channel-averaged latent clips for the spectral analysis
    (the paper's Pexels clips and Wan VAE are not available).

    Each frame is a sum of smoothed random fields at several spatial scales:
    level s is white noise box-filtered with half-width w_s (wider = lower
    spatial frequencies), evolving over frames as an AR(1) process with
    coefficient rho_s (wider = slower), so coarse structure stays
    correlated over longer lags than fine structure.  ``clip()`` returns a
    float32 tensor [frames][H][W]."""

    def __init__(self, seed: int, frames: int, height: int, width: int, device="cpu",
                 widths=(0, 1, 3, 7, 15), rhos=(0.5, 0.8, 0.93, 0.98, 0.995)):
        import torch
        self.torch = torch
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed)
        self.shape = (frames, height, width)
        self.device = device
        self.widths, self.rhos = widths, rhos

    def _box(self, x, w):
        """Separable box filter of half-width w (replicate edges), on [T][H][W]."""
        if w == 0:
            return x
        torch = self.torch
        k = torch.ones(1, 1, 2 * w + 1, dtype=x.dtype, device=x.device) / (2 * w + 1)
        T, H, W = x.shape
        y = torch.nn.functional.pad(x.reshape(T * H, 1, W), (w, w), mode="replicate")
        y = torch.nn.functional.conv1d(y, k).reshape(T, H, W).transpose(1, 2)
        y = torch.nn.functional.pad(y.reshape(T * W, 1, H), (w, w), mode="replicate")
        return torch.nn.functional.conv1d(y, k).reshape(T, W, H).transpose(1, 2).contiguous()

    def clip(self):
        torch = self.torch
        T, H, W = self.shape
        z = torch.zeros(self.shape, dtype=torch.float32, device=self.device)
        for w, rho in zip(self.widths, self.rhos):
            e = torch.randn(self.shape, generator=self.gen, device=self.device, dtype=torch.float32)
            a = torch.empty_like(e)
            a[0] = e[0]
            b = float(np.sqrt(1.0 - rho * rho))
            for t in range(1, T):
                a[t] = rho * a[t - 1] + b * e[t]
            f = self._box(a, w)
            z += f / f.std()
        return z

"""Smooth-field + noise Q/K/V generator for attention over a (T, Hs, Ws) token grid.

Real video-DiT activations are spatio-temporally continuous (paper §2.1: the
latent keeps the (T, H, W) structure and is flattened to one token sequence),
which is what makes 3D block summaries informative. The datasets and weights the
paper measures on are not available, so inputs are synthetic:

    X[b, h, n, c] = noise * eps + gain_X * F[b, h, n, c]
    F[c](t, y, x) = 1/n_waves * sum_m cos(2*pi*<omega_m, (t, y, x)> + phi[m, c])

with eps ~ N(0, 1) i.i.d. Q and K of one head share the wave vectors and phases
(so pooled Q.K is a stationary kernel peaked at zero displacement, i.e. local
attention with some periodic long-range echoes); V draws its own phases.
omega_m = f_h * (u_m scaled per axis by `aniso`), u_m uniform on the unit sphere,
f_h the head's bandwidth in cycles per token.

Token order is T-major raster: n = (t * Hs + y) * Ws + x.
"""
from __future__ import annotations

import math

import numpy as np
import torch


def bf16_round(x: torch.Tensor) -> torch.Tensor:
    """Round to bfloat16 with round-to-nearest-even (torch's cast)."""
    return x.to(torch.bfloat16)


def _wave_params(rng: np.random.Generator, n_waves: int, d: int, freq: float, aniso):
    u = rng.standard_normal((n_waves, 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    omega = freq * u * np.asarray(aniso, dtype=np.float64)[None, :]
    phi_qk = rng.uniform(0.0, 2.0 * math.pi, size=(n_waves, d))
    phi_v = rng.uniform(0.0, 2.0 * math.pi, size=(n_waves, d))
    return omega, phi_qk, phi_v


def _field(coords: np.ndarray, omega: np.ndarray, phi: np.ndarray) -> np.ndarray:
    """F[n, c] = mean_m cos(theta_m[n] + phi[m, c]) as one [N, 2M] x [2M, d] product."""
    theta = 2.0 * math.pi * coords @ omega.T                     # [N, M]
    basis = np.concatenate([np.cos(theta), -np.sin(theta)], 1)  # [N, 2M]
    coef = np.concatenate([np.cos(phi), np.sin(phi)], 0)         # [2M, d]
    return (basis @ coef) / omega.shape[0]


def grid_coords(T: int, Hs: int, Ws: int) -> np.ndarray:
    t, y, x = np.meshgrid(np.arange(T), np.arange(Hs), np.arange(Ws), indexing="ij")
    return np.stack([t.ravel(), y.ravel(), x.ravel()], 1).astype(np.float64)


def smooth_field_qkv(B: int, H: int, T: int, Hs: int, Ws: int, d: int, *,
                     seed: int = 0, gain_qk=1.0, freqs=0.05, noise: float = 0.5,
                     n_waves: int = 4, aniso=(1.0, 1.0, 1.0), device="cpu",
                     dtype=torch.float32):
    """Return (Q, K, V), each [B, H, N, d] of `dtype` on `device`.

    gain_qk, freqs and aniso may be scalars or per-head sequences (length H;
    aniso entries are 3-tuples). The small parameters come from numpy's PCG64
    seeded with `seed`; the i.i.d. noise from a torch generator on `device`
    seeded with `seed`, so a (seed, device) pair always gives the same tensors.
    """
    N = T * Hs * Ws
    gains = np.broadcast_to(np.asarray(gain_qk, dtype=np.float64), (H,))
    fr = np.broadcast_to(np.asarray(freqs, dtype=np.float64), (H,))
    an = np.asarray(aniso, dtype=np.float64)
    an = np.broadcast_to(an if an.ndim == 2 else an[None, :], (H, 3))
    rng = np.random.default_rng(seed)
    coords = grid_coords(T, Hs, Ws)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    out = []
    fq = torch.empty((B, H, N, d), dtype=torch.float32)
    fv = torch.empty((B, H, N, d), dtype=torch.float32)
    for b in range(B):
        for h in range(H):
            omega, phi_qk, phi_v = _wave_params(rng, n_waves, d, fr[h], an[h])
            fq[b, h] = torch.from_numpy((gains[h] * _field(coords, omega, phi_qk)).astype(np.float32))
            fv[b, h] = torch.from_numpy(_field(coords, omega, phi_v).astype(np.float32))
    fq = fq.to(device)
    fv = fv.to(device)
    for f in (fq, fq, fv):
        eps = torch.randn((B, H, N, d), generator=gen, device=device, dtype=torch.float32)
        out.append((noise * eps + f).to(dtype))
    return tuple(out)

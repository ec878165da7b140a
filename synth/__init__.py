"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This module holds random-number plumbing only: it draws tensors of given
shapes from seeded numpy generators.  It contains none of the method's
arithmetic (no model, no interpolation weights, no aggregation), so the
oracle and the HIP path can both take their inputs from here without
sharing any code that computes a result.

Recipe (per workload):
  * parameters: every weight and bias ~ N(0, std) with std = 0.02; the
    per-head query/key normalisation gains are 1 + N(0, std) (a gain drawn
    around zero would zero the attention logits);
  * latents, text embeddings, token streams: N(0, 1);
  * per-step upstream gradients s_j = A * g_j with A ~ N(0, 1) one scalar
    advantage per sample and g_j ~ N(0, 1) (GRPO advantages scale the whole
    per-step gradient of a rollout);
  * timesteps: the unshifted uniform grid t_k = 1 - k/T, k = 0..T-1.
"""
from __future__ import annotations

import numpy as np

THETA_SEED = 42
DATA_SEED = 12627


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def theta(layout, seed: int = THETA_SEED, std: float = 0.02, gain_std: float | None = None,
          dtype=np.float64, total: int | None = None) -> np.ndarray:
    """Flat parameter vector for ``layout``: iterable of (name, offset, numel).

    ``total`` is the padded length (default: end of the last tensor).  Padding
    between tensors is zero.  Names ending in ``_gain`` are drawn as
    1 + N(0, gain_std) (gain_std defaults to std)."""
    entries = list(layout)
    if total is None:
        total = max(off + n for _, off, n in entries) if entries else 0
    out = np.zeros(total, dtype=dtype)
    g = rng(seed)
    gs = std if gain_std is None else gain_std
    for name, off, n in entries:
        if name.endswith("_gain"):
            out[off:off + n] = 1.0 + gs * g.standard_normal(n)
        else:
            out[off:off + n] = std * g.standard_normal(n)
    return out


def normal(shape, seed: int, scale: float = 1.0, dtype=np.float64) -> np.ndarray:
    return (scale * rng(seed).standard_normal(shape)).astype(dtype)


def uniform_grid(T: int) -> np.ndarray:
    """t_k = 1 - k/T for k = 0..T-1 (all in (0, 1])."""
    return np.array([1.0 - k / T for k in range(T)], dtype=np.float64)


def upstream_grads(W: int, shape, seed: int, batch: int = 1, dtype=np.float64):
    """W per-step upstream gradients s_j = A_b * g_j (A_b ~ N(0,1) per sample b).

    ``shape`` is the per-step output shape whose leading axis is the batch."""
    g = rng(seed)
    adv = g.standard_normal(batch)
    out = []
    for _ in range(W):
        gj = g.standard_normal(shape)
        scale = adv.reshape((batch,) + (1,) * (len(shape) - 1))
        out.append((gj * scale).astype(dtype))
    return out, adv


def orthonormal_rows(k: int, n: int, seed: int) -> np.ndarray:
    """k exactly orthonormal rows of length n (fp64 modified Gram-Schmidt, twice)."""
    g = rng(seed)
    m = g.standard_normal((k, n))
    for _ in range(2):
        for i in range(k):
            for j in range(i):
                m[i] -= np.dot(m[i], m[j]) * m[j]
            m[i] /= np.linalg.norm(m[i])
    return m


def hidden_profile(W: int, n: int, rho: float, seed: int) -> np.ndarray:
    """W per-step hidden-state vectors h_j = sqrt(rho) u + sqrt(1-rho) e_j.

    With u, e_0..e_{W-1} exactly orthonormal, every pair has cosine rho."""
    basis = orthonormal_rows(W + 1, n, seed)
    u, e = basis[0], basis[1:]
    return np.sqrt(rho) * u[None, :] + np.sqrt(1.0 - rho) * e


def device_normal(shape, seed: int, std: float = 1.0, dtype=None, device="cuda"):
    """N(0, std^2) drawn on the device with a seeded torch generator (for
    full-size workloads, where host generation would dominate set-up time)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x if dtype is None else x.to(dtype)

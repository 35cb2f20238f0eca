"""Offline-fusion identities of the two cache paths -- oracle (test infrastructure).

Sec. 3.1 ("Path-Specific Offline-Fusible Transformation Spaces") and
Appendix C.1-C.2 ("Content-Path Fusion", "RoPE-Path Fusion").  Row-vector
convention throughout (a projection is ``h @ W``).

Content path.  The cached latent is ``c = u Gamma`` with ``u`` the weightless
RMSNorm of the producing projection's output and ``Gamma = Diag(gamma)``.
With an orthogonal ``R_C`` and a positive diagonal ``S_C`` the cache becomes
``z_C = u R_C S_C``; the producing projection absorbs ``R_C`` (weightless
RMSNorm commutes with it), the normalization scale becomes ``S_C`` and every
consumer ``W_b`` becomes ``S_C^-1 R_C^T Gamma W_b``, so ``z_C W_b' = c W_b``.

RoPE path (Proposition 1).  With ``R_P = blockdiag(R_i)``, ``R_i`` in SO(2) on
frequency pair ``i``, and ``S_P = blockdiag(s_i I_2)``, the reciprocal
transform ``Q' = Q R_P S_P^-1``, ``K' = K R_P S_P`` keeps ``Q K^T``, and both
factors commute with every RoPE rotation on the same pairs, so they fold into
the pre-RoPE projections ``W_Q' = W_Q R_P S_P^-1``, ``W_K' = W_K R_P S_P``.

RoPE layout used here (the synthetic inputs' convention): pair ``i`` is
channels ``(2i, 2i+1)`` rotated by angle ``t * base**(-2i/d)`` at position
``t``.

Everything is fp64 numpy.  The learning of ``R_C, S_C, R_P, S_P`` is out of
scope (it needs model weights and calibration data); the identities hold for
any admissible transform, so random ones are used.  Shares no code with the
GPU library.
"""
from __future__ import annotations

import numpy as np


def rmsnorm_weightless(x: np.ndarray, eps: float = 0.0) -> np.ndarray:
    """``x / sqrt(mean(x^2) + eps)`` over the last axis."""
    x = np.asarray(x, np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def random_orthogonal(rng: np.random.Generator, d: int) -> np.ndarray:
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))[None, :]


# ---- content path ---------------------------------------------------------

def content_latent(h: np.ndarray, gamma: np.ndarray, eps: float = 0.0) -> np.ndarray:
    """The original cached latent ``c = RMSNorm_1(h) Gamma``."""
    return rmsnorm_weightless(h, eps) * np.asarray(gamma, np.float64)[None, :]


def fuse_content(W_a: np.ndarray, gamma: np.ndarray, consumers, R_C: np.ndarray, s_C: np.ndarray):
    """Offline reparameterization of the content path.

    Returns ``(W_a', gamma', [W_b', ...])`` with ``W_a' = W_a R_C``,
    ``gamma' = s_C`` and ``W_b' = S_C^-1 R_C^T Gamma W_b``.
    """
    gamma = np.asarray(gamma, np.float64)
    s_C = np.asarray(s_C, np.float64)
    W_a2 = np.asarray(W_a, np.float64) @ R_C
    fused = [(1.0 / s_C)[:, None] * (R_C.T @ (gamma[:, None] * np.asarray(W_b, np.float64))) for W_b in consumers]
    return W_a2, s_C.copy(), fused


# ---- RoPE path ------------------------------------------------------------

def rope_angles(positions, d: int, base: float = 10000.0) -> np.ndarray:
    """Angle of frequency pair ``i`` at each position: ``t * base**(-2i/d)``."""
    i = np.arange(d // 2, dtype=np.float64)
    return np.asarray(positions, np.float64)[:, None] * base ** (-2.0 * i / d)[None, :]


def apply_rope(x: np.ndarray, positions, base: float = 10000.0) -> np.ndarray:
    """Rotate pair ``(2i, 2i+1)`` of row ``r`` by its angle at ``positions[r]``."""
    x = np.asarray(x, np.float64)
    a = rope_angles(positions, x.shape[-1], base)
    c, s = np.cos(a), np.sin(a)
    out = np.empty_like(x)
    out[:, 0::2] = x[:, 0::2] * c - x[:, 1::2] * s
    out[:, 1::2] = x[:, 0::2] * s + x[:, 1::2] * c
    return out


def pair_transform(angles: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """``R_P S_P`` as a dense matrix: pair ``i`` rotated by ``angles[i]``, scaled by ``scales[i]``.

    Row-vector convention: ``x @ M`` rotates each pair of ``x`` by its angle.
    """
    n = len(angles)
    M = np.zeros((2 * n, 2 * n))
    for i, (t, s) in enumerate(zip(angles, scales)):
        c, sn = np.cos(t), np.sin(t)
        M[2 * i:2 * i + 2, 2 * i:2 * i + 2] = s * np.array([[c, sn], [-sn, c]])
    return M


def fuse_rope(W_Q: np.ndarray, W_K: np.ndarray, angles: np.ndarray, scales: np.ndarray):
    """Reciprocal pre-RoPE fusion: ``W_Q' = W_Q R_P S_P^-1``, ``W_K' = W_K R_P S_P``."""
    RS = pair_transform(angles, scales)
    RSinv = pair_transform(angles, 1.0 / np.asarray(scales, np.float64))
    return np.asarray(W_Q, np.float64) @ RSinv, np.asarray(W_K, np.float64) @ RS

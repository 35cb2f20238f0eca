"""Absorbed dual-path MLA decode attention -- oracle (test infrastructure).

Sec. 2.1, eq. mla_compact: per head ``h``::

    S_h = tau * (Qbar_C,h C^T + Q_P,h K_P^T) + M_attn,   A_h = softmax(S_h)

and the kernel boundary stops at the latent aggregation ``O_h = A_h C``
(value/output projections keep their own boundary, Appendix C.5, "Cache update
and tile reuse").  Everything here is fp64, computed from the fp32
reconstructed cache and the bf16 queries widened exactly.

Causal mask (reading 12 in the design doc): a sequence of length ``L`` whose last
``s_q`` tokens are the queries lets query ``i`` see keys ``t <= L - s_q + i``.

Chunk partials and their merge follow Appendix C.5, "Global attention
normalization": a chunk ``j`` of keys yields its maximum logit ``m_j``, its
exponential sum ``s_j`` and its unnormalised weighted latent sum ``o_j``; the
global result is ``m = max m_j``, ``s = sum e^{m_j-m} s_j``,
``o = sum e^{m_j-m} o_j``, ``O = o / s``.  A chunk with no valid key is
``(-inf, 0, 0)`` and is skipped (reading 11).

Pure numpy; shares no code with the GPU library.
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits) -> np.ndarray:
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def logits(q_lat, q_rope, c_hat, kr_hat, tau):
    """``z[r, t] = tau * (q_lat[r].c_hat[t] + q_rope[r].kr_hat[t])`` in fp64."""
    q_lat = np.asarray(q_lat, np.float64)
    q_rope = np.asarray(q_rope, np.float64)
    c = np.asarray(c_hat, np.float64)
    k = np.asarray(kr_hat, np.float64)
    return float(tau) * (q_lat @ c.T + q_rope @ k.T)


def _valid(limits, L):
    limits = np.asarray(limits, np.int64).reshape(-1, 1)
    return np.arange(L, dtype=np.int64)[None, :] < limits


def attend(q_lat, q_rope, c_hat, kr_hat, tau, limits):
    """Exact softmax attention for rows ``r`` over keys ``t < limits[r]``.

    Returns ``(out [R, d_c], lse [R])`` with ``lse`` the natural-log
    log-sum-exp of the scaled logits.  Every row needs at least one valid key.
    """
    z = logits(q_lat, q_rope, c_hat, kr_hat, tau)
    valid = _valid(limits, z.shape[1])
    if not np.all(valid.any(axis=1)):
        raise ValueError("every query row needs at least one valid key")
    z = np.where(valid, z, -np.inf)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1, keepdims=True)
    out = (e @ np.asarray(c_hat, np.float64)) / s
    lse = (m + np.log(s))[:, 0]
    return out, lse


def chunk_partials(q_lat, q_rope, c_hat, kr_hat, tau, limits, bounds):
    """Per-chunk ``(m_j, s_j, o_j)`` for key ranges ``bounds = [(start, end), ...]``.

    Shapes: ``m, s`` are ``[J, R]``, ``o`` is ``[J, R, d_c]``.
    """
    z = logits(q_lat, q_rope, c_hat, kr_hat, tau)
    valid = _valid(limits, z.shape[1])
    c = np.asarray(c_hat, np.float64)
    R = z.shape[0]
    J = len(bounds)
    m = np.full((J, R), -np.inf)
    s = np.zeros((J, R))
    o = np.zeros((J, R, c.shape[1]))
    for j, (a, b) in enumerate(bounds):
        zj = np.where(valid[:, a:b], z[:, a:b], -np.inf)
        for r in range(R):
            if not np.isfinite(zj[r]).any():
                continue                      # empty chunk for this row: (-inf, 0, 0)
            m[j, r] = zj[r].max()
            e = np.exp(zj[r] - m[j, r])
            s[j, r] = e.sum()
            o[j, r] = e @ c[a:b]
    return m, s, o


def merge(m, s, o):
    """Global normalisation of chunk partials; returns ``(out [R, d], lse [R])``."""
    m = np.asarray(m, np.float64)
    s = np.asarray(s, np.float64)
    o = np.asarray(o, np.float64)
    J, R = m.shape
    out = np.zeros((R, o.shape[2]))
    lse = np.zeros(R)
    for r in range(R):
        live = [j for j in range(J) if np.isfinite(m[j, r])]
        if not live:
            raise ValueError("row without any valid key")
        mm = max(m[j, r] for j in live)
        ss = sum(np.exp(m[j, r] - mm) * s[j, r] for j in live)
        oo = sum(np.exp(m[j, r] - mm) * o[j, r] for j in live)
        out[r] = oo / ss
        lse[r] = mm + np.log(ss)
    return out, lse


def decode_limits(L: int, s_q: int, H: int) -> np.ndarray:
    """Visible-key count of every (query token i, head h) row, row-major in (i, h)."""
    return np.repeat(np.arange(L - s_q + 1, L + 1, dtype=np.int64), H)


def decode_sequence(q_lat_bits, q_rope_bits, c_hat, kr_hat, tau, heads=None):
    """Decode attention of one sequence.

    ``q_lat_bits [s_q, H, d_c]`` and ``q_rope_bits [s_q, H, d_r]`` are bf16 bit
    patterns; ``c_hat [L, d_c]`` and ``kr_hat [L, d_r]`` the reconstructed
    cache.  ``heads`` optionally restricts the computation to some heads.
    Returns ``(out [s_q, Hsel, d_c], lse [s_q, Hsel])`` in fp64.
    """
    ql = bf16_bits_to_f64(q_lat_bits)
    qr = bf16_bits_to_f64(q_rope_bits)
    s_q, H = ql.shape[:2]
    if heads is not None:
        ql = ql[:, heads]
        qr = qr[:, heads]
    Hs = ql.shape[1]
    L = np.asarray(c_hat).shape[0]
    out, lse = attend(ql.reshape(s_q * Hs, -1), qr.reshape(s_q * Hs, -1), c_hat, kr_hat,
                      tau, decode_limits(L, s_q, Hs))
    return out.reshape(s_q, Hs, -1), lse.reshape(s_q, Hs)

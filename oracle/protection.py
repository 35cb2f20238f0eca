"""BF16 protection of sink and recent tokens -- oracle (test infrastructure).

Sec. 3.3 and Appendix C.5 ("BF16 protection and cache lifecycle", "Global
attention normalization", "Storage layout").  Besides the packed copy of every
token, the fused writer keeps the pre-quantization bf16 content latent and RoPE
key of the first ``sink`` tokens and of the ``recent`` most recent tokens.  For
a sequence of ``L`` cached tokens (positions ``0 .. L-1``) the protected set is

    P_L = {0, ..., min(sink, L) - 1}  U  {max(0, L - recent), ..., L - 1}

with overlapping positions counted once (the paper's policy: sink = 4,
recent = 128).  Attention uses exactly one representation per token -- the
bf16 values for positions in ``P_L``, the values reconstructed from the packed
copy for every other position -- and all visible tokens share one softmax; a
token that leaves the recent window falls back to the packed copy written when
it was inserted.  No token is dropped or masked by the policy.

Protection buffer.  The paper fixes its size, ``sink + recent`` rows of
``d_c + d_r`` bf16 values per sequence and layer, not its order; the library's
order (reading 17 in the design doc) is: row ``p`` holds position ``p < sink``, row
``sink + (p - sink) mod recent`` holds position ``p >= sink`` -- a ring, in
which the token entering the recent window overwrites the one leaving it.  A
row is ``[c_kv (d_c) | k_rope (d_r)]`` copied bit for bit.

Writer rule for one append call: the tokens of a sequence whose length after
the call is ``L`` are written to the buffer when ``p < sink`` or
``p >= L - recent``; a long prefill thus writes only the rows that are
protected once it is done, and no two of its tokens share a row.

Pure numpy; shares no code with the GPU library.
"""
from __future__ import annotations

import numpy as np

from . import attention as at
from . import paged_cache as pc

SINK = 4
RECENT = 128


def protected_positions(L: int, sink: int = SINK, recent: int = RECENT) -> np.ndarray:
    """Sorted positions of ``P_L`` (the set union of the sink and the window)."""
    head = np.arange(min(sink, L), dtype=np.int64)
    tail = np.arange(max(0, L - recent), L, dtype=np.int64)
    return np.union1d(head, tail)


def protected_mask(L: int, sink: int = SINK, recent: int = RECENT) -> np.ndarray:
    m = np.zeros(L, dtype=bool)
    m[protected_positions(L, sink, recent)] = True
    return m


def buffer_row(p: int, sink: int = SINK, recent: int = RECENT) -> int:
    """Buffer row of position ``p`` (the library's ring order)."""
    if p < sink:
        return p
    if recent <= 0:
        raise ValueError("position past the sink with no recent window")
    return sink + (p - sink) % recent


def write_protection(buf: np.ndarray, positions, seq_len: int, c_kv_bits, k_rope_bits,
                     sink: int = SINK, recent: int = RECENT) -> None:
    """One append call's protection writes for ONE sequence.

    ``buf`` is the sequence's ``[sink + recent, d_c + d_r]`` uint16 buffer;
    ``positions`` the appended tokens' positions, ``seq_len`` the sequence's
    length after the call, ``c_kv_bits``/``k_rope_bits`` their bf16 rows.
    """
    c = np.asarray(c_kv_bits, np.uint16)
    k = np.asarray(k_rope_bits, np.uint16)
    for i, p in enumerate(np.asarray(positions, np.int64).reshape(-1)):
        if p < sink or (p >= seq_len - recent and p < seq_len):
            buf[buffer_row(int(p), sink, recent)] = np.concatenate([c[i], k[i]])


def read_protection(buf: np.ndarray, L: int, d_c: int = 512, sink: int = SINK, recent: int = RECENT):
    """The bf16 rows of ``P_L`` as stored: ``(positions, c_kv bits, k_rope bits)``."""
    pos = protected_positions(L, sink, recent)
    rows = np.asarray([buf[buffer_row(int(p), sink, recent)] for p in pos], np.uint16).reshape(len(pos), -1)
    return pos, rows[:, :d_c], rows[:, d_c:]


def representation(fmt: pc.CacheFormat, c_kv_bits, k_rope_bits, sink: int = SINK, recent: int = RECENT):
    """The values attention uses for each of the ``L`` tokens (fp64).

    bf16 values (exact) for positions in ``P_L``; for every other position the
    reconstruction from the packed cache (fp32 quantize/dequantize of
    Appendix C.4, as :func:`oracle.paged_cache.encode_sequence_dense`).
    """
    c_kv_bits = np.asarray(c_kv_bits, np.uint16).reshape(-1, fmt.d_c)
    k_rope_bits = np.asarray(k_rope_bits, np.uint16).reshape(-1, fmt.d_r)
    L = c_kv_bits.shape[0]
    c_hat, kr_hat = pc.encode_sequence_dense(fmt, c_kv_bits, k_rope_bits)
    keep = protected_mask(L, sink, recent)[:, None]
    c = np.where(keep, at.bf16_bits_to_f64(c_kv_bits), c_hat.astype(np.float64))
    k = np.where(keep, at.bf16_bits_to_f64(k_rope_bits), kr_hat.astype(np.float64))
    return c, k


def decode_sequence_protected(fmt: pc.CacheFormat, q_lat_bits, q_rope_bits, c_kv_bits, k_rope_bits, tau,
                              sink: int = SINK, recent: int = RECENT, heads=None):
    """Decode attention of one sequence under the protection policy.

    One softmax over all visible tokens, each in its single representation;
    causal reading and shapes as :func:`oracle.attention.decode_sequence`.
    """
    c, k = representation(fmt, c_kv_bits, k_rope_bits, sink, recent)
    return at.decode_sequence(q_lat_bits, q_rope_bits, c, k, tau, heads=heads)


def region_partials(fmt: pc.CacheFormat, q_lat_bits, q_rope_bits, c_kv_bits, k_rope_bits, tau,
                    sink: int = SINK, recent: int = RECENT):
    """Partials ``(m_j, s_j, o_j)`` of the two regions processed separately.

    Region 0 is the packed history (reconstructed values), region 1 the
    protected tokens (bf16 values); each is attended on its own, as in
    Appendix C.5, "Global attention normalization".  Merged by
    :func:`oracle.attention.merge` they give the single softmax.
    """
    ql = at.bf16_bits_to_f64(q_lat_bits)
    qr = at.bf16_bits_to_f64(q_rope_bits)
    s_q, H = ql.shape[:2]
    c_kv_bits = np.asarray(c_kv_bits, np.uint16).reshape(-1, fmt.d_c)
    k_rope_bits = np.asarray(k_rope_bits, np.uint16).reshape(-1, fmt.d_r)
    L = c_kv_bits.shape[0]
    keep = protected_mask(L, sink, recent)
    c_hat, kr_hat = pc.encode_sequence_dense(fmt, c_kv_bits, k_rope_bits)
    lim = at.decode_limits(L, s_q, H)
    ms, ss, os_ = [], [], []
    for sel, c, k in ((~keep, c_hat, kr_hat),
                      (keep, at.bf16_bits_to_f64(c_kv_bits), at.bf16_bits_to_f64(k_rope_bits))):
        pos = np.nonzero(sel)[0]
        # visible keys of a row are the region's positions below its limit
        sub_lim = np.searchsorted(pos, lim, side="left")
        m, s, o = at.chunk_partials(ql.reshape(s_q * H, -1), qr.reshape(s_q * H, -1),
                                    np.asarray(c, np.float64)[pos], np.asarray(k, np.float64)[pos], tau,
                                    sub_lim, [(0, len(pos))])
        ms.append(m[0])
        ss.append(s[0])
        os_.append(o[0])
    return np.stack(ms), np.stack(ss), np.stack(os_)

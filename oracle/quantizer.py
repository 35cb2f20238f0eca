"""Affine asymmetric per-token group quantizer -- oracle (test infrastructure).

Follows Appendix C.4, "Affine group quantization": every token is quantized on
its own, in groups of 64 consecutive coordinates.  For ``b`` bits,
``m = 2**b - 1`` and, per group with extrema ``xmin``, ``xmax``::

    s = max(xmax - xmin, 1e-8) / m
    z = clip(round(-xmin / s), 0, m)
    q = clip(round(x / s + z), 0, m)
    x_hat = s * (q - z)

with round-half-to-even and no special case for constant groups.  Native
execution keeps the stored (rounded) scale and dequantizes with it (same
paragraph, last sentence).

Readings taken where the paper leaves a choice (all listed in the design doc):
  * inputs are bf16, widened exactly to fp32; every step is one IEEE fp32
    operation with round-half-to-even, in the order written above (a true
    division, then an addition: two roundings, no fused multiply-add);
  * the constant 1e-8 is the fp32 value nearest to it;
  * the zero-point is the integer ``clip(round(-xmin/s), 0, m)``; when
    ``-xmin/s`` rounds to -0 it is stored as +0;
  * codes come from the unrounded fp32 scale ``s``; the stored scale is
    ``fp16(s)`` (round-half-to-even, subnormals kept) and the stored zero is
    ``fp16(z)``, which is exact;
  * dequantization is ``fp16scale * (q - fp16zero)`` evaluated in fp32
    (``q - z`` is exact, so this is a single rounding);
  * the paper's own storage (same paragraph, last sentence): content scales
    in BF16 (``bf16(s)``, round-half-to-even), RoPE scales in FP32 (``s``
    itself); the zero-point, whose dtype the paper leaves open, as an unsigned
    byte (exact: an integer in ``[0, m]``).  Dequantization multiplies by the
    stored scale the same way.

Codes are packed into little-endian 32-bit words of ``32 / bits`` consecutive
channels (8 at 4 bits, 16 at 2 bits), stored as the word's four bytes.  Inside
a word, channel ``2i`` occupies bits ``[bits*i, bits*(i+1))`` and channel
``2i+1`` the same bits of the upper 16-bit half, i.e. bits
``[16 + bits*i, 16 + bits*(i+1))``.  For 4 bits the word of channels 0..7
holds channels 0, 2, 4, 6 in its low half (bytes 0-1) and 1, 3, 5, 7 in its
high half (bytes 2-3); for 2 bits the low half holds channels 0, 2, ..., 14
and the high half 1, 3, ..., 15.  The paper fixes only the byte count per
token; this order lets a decoder take a channel pair with one shift and one
mask (:func:`pack_codes`, :func:`unpack_codes`).

Pure numpy; shares no code with the GPU library.
"""
from __future__ import annotations

import numpy as np

GROUP = 64
EPS = np.float32(1e-8)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def levels(bits: int) -> np.float32:
    """``m = 2**b - 1`` as fp32 (Appendix C.4)."""
    if bits not in (2, 4):
        raise ValueError(f"unsupported bit width {bits}")
    return np.float32((1 << bits) - 1)


def quantize_groups(x: np.ndarray, bits: int):
    """Quantize the last axis of ``x`` (float32, length 64 = one group).

    Returns ``(q, s, z)``: integer codes (uint8, same shape as ``x``), the
    unrounded fp32 scale and the fp32 zero-point per group (shape ``x.shape[:-1]``).
    """
    x = np.asarray(x, dtype=np.float32)
    if x.shape[-1] != GROUP:
        raise ValueError("last axis must be one group of 64 coordinates")
    m = levels(bits)
    xmin = x.min(axis=-1)
    xmax = x.max(axis=-1)
    r = (xmax - xmin).astype(np.float32)                       # fp32 subtraction
    s = (np.maximum(r, EPS) / m).astype(np.float32)            # true fp32 division
    z = np.clip(np.rint((-xmin) / s), np.float32(0), m).astype(np.float32)
    z = (z + np.float32(0)).astype(np.float32)   # the integer zero-point: +0, never -0
    t = (x / s[..., None]).astype(np.float32)                  # rounding 1: divide
    t = (t + z[..., None]).astype(np.float32)                  # rounding 2: add
    q = np.clip(np.rint(t), np.float32(0), m).astype(np.uint8)
    return q, s, z


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), returned as
    float32 values; finite inputs only."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)) << np.uint32(16)
    return r.astype(np.uint32).view(np.float32)


def stored_meta_paper(s: np.ndarray, z: np.ndarray, rope: bool):
    """The paper's stored scale (BF16 for the content path, FP32 for the RoPE
    path) and the zero-point as an unsigned byte."""
    s = np.asarray(s, dtype=np.float32)
    return (s.copy() if rope else f32_to_bf16(s)), np.asarray(z, dtype=np.float32).astype(np.uint8)


def stored_meta(s: np.ndarray, z: np.ndarray):
    """Stored fp16 scale and zero-point (round-half-to-even, subnormals kept)."""
    return (np.asarray(s, dtype=np.float32).astype(np.float16),
            np.asarray(z, dtype=np.float32).astype(np.float16))


def dequantize(q: np.ndarray, scale16: np.ndarray, zero16: np.ndarray) -> np.ndarray:
    """``x_hat = scale * (q - zero)`` in fp32 with the stored metadata.

    ``q`` has a trailing group axis of 64; ``scale16``/``zero16`` one value per
    group, as stored (fp16, or the paper's bf16-valued / fp32 scales and byte
    zero-points); every stored value widens exactly to fp32.
    """
    sc = np.asarray(scale16).astype(np.float32)[..., None]
    ze = np.asarray(zero16).astype(np.float32)[..., None]
    d = (np.asarray(q).astype(np.float32) - ze).astype(np.float32)   # exact: small integers
    return (sc * d).astype(np.float32)


def pack_codes(q: np.ndarray, bits: int) -> np.ndarray:
    """Pack integer codes along the last axis into little-endian 32-bit words of
    32 / bits consecutive channels (the library's byte layout): of the channel
    pair (2i, 2i+1) of a word, channel 2i occupies bits [bits*i, bits*(i+1))
    of the word and channel 2i+1 the same bits of its upper 16-bit half."""
    q = np.asarray(q, dtype=np.uint8)
    per = 32 // bits
    if q.shape[-1] % per:
        raise ValueError("channel count must fill whole 32-bit words")
    if np.any(q > (1 << bits) - 1):
        raise ValueError("code out of range")
    q = q.reshape(q.shape[:-1] + (q.shape[-1] // per, per)).astype(np.uint32)
    word = np.zeros(q.shape[:-1], dtype=np.uint32)
    for i in range(per // 2):
        word |= q[..., 2 * i] << np.uint32(bits * i)
        word |= q[..., 2 * i + 1] << np.uint32(16 + bits * i)
    out = word.astype("<u4").view(np.uint8)
    return out.reshape(q.shape[:-2] + (q.shape[-2] * 4,))


def unpack_codes(packed: np.ndarray, bits: int) -> np.ndarray:
    """Inverse of :func:`pack_codes`."""
    packed = np.ascontiguousarray(np.asarray(packed, dtype=np.uint8))
    if packed.shape[-1] % 4:
        raise ValueError("packed codes come in whole 32-bit words")
    word = packed.view("<u4").astype(np.uint32)
    mask = np.uint32((1 << bits) - 1)
    per = 32 // bits
    parts = []
    for i in range(per // 2):
        parts.append((word >> np.uint32(bits * i)) & mask)
        parts.append((word >> np.uint32(16 + bits * i)) & mask)
    out = np.stack(parts, axis=-1).astype(np.uint8)
    return out.reshape(word.shape[:-1] + (word.shape[-1] * per,))


def quantize_token_path(x_bits: np.ndarray, bits: int, meta: str = "fp16", rope: bool = False):
    """Quantize one cache path for a batch of tokens.

    ``x_bits``: bf16 bit patterns, shape ``[n, d]`` with ``d % 64 == 0``.
    Returns ``(packed [n, d*bits/8] uint8, scale [n, d/64], zero [n, d/64])``
    with the metadata as stored: fp16 scale and zero (``meta="fp16"``), or the
    paper's bf16 (content) / fp32 (RoPE, ``rope=True``) scale and byte zero
    (``meta="paper"``).
    """
    x = bf16_bits_to_f32(x_bits)
    n, d = x.shape
    if d % GROUP:
        raise ValueError("path width must be a multiple of the group size")
    q, s, z = quantize_groups(x.reshape(n, d // GROUP, GROUP), bits)
    if meta == "paper":
        sm, zm = stored_meta_paper(s, z, rope)
    elif meta == "fp16":
        sm, zm = stored_meta(s, z)
    else:
        raise ValueError(meta)
    return pack_codes(q.reshape(n, d), bits), sm, zm


def dequantize_token_path(packed: np.ndarray, scale16: np.ndarray, zero16: np.ndarray,
                          bits: int) -> np.ndarray:
    """Dequantize packed codes ``[n, d*bits/8]`` back to fp32 ``[n, d]``."""
    q = unpack_codes(packed, bits)
    n, d = q.shape
    xh = dequantize(q.reshape(n, d // GROUP, GROUP), scale16, zero16)
    return xh.reshape(n, d)

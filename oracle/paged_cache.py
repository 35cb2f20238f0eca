"""Packed, paged dual-path cache -- oracle (test infrastructure).

Appendix C.5 ("Cache update and tile reuse", "Storage layout"): the writer
quantizes the content latent and the RoPE key of every incoming token, packs
the integer codes and inserts them at the token's slot in a page; attention
later gathers pages, unpacks codes and reconstructs both paths from the stored
scales and zero-points.  The paper fixes the quantizer and the page size (64
tokens) but not the byte order inside a page; this module states the one the
library uses (reading 8 in the design doc) and builds it byte by byte.

One page of ``P`` tokens holds four token-major regions, in this order::

    codes_c[P][d_c * c_bits / 8]      packed content codes
    codes_r[P][d_r * r_bits / 8]      packed RoPE-key codes
    meta_c [P][d_c / 64][2] fp16      (scale, zero) per content group
    meta_r [P][d_r / 64][2] fp16      (scale, zero) per RoPE group

and the page size in bytes is rounded up to a multiple of 256.  A slot is
``page * P + offset``; a negative slot means "do not store this token".
For ``d_c=512, d_r=64, P=64`` this is 20 736 B per page with 4-bit content
(324 B per token) and 12 544 B with 2-bit content (196 B per token).

Pure numpy; shares no code with the GPU library.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import quantizer as qz


@dataclass(frozen=True)
class CacheFormat:
    d_c: int = 512
    d_r: int = 64
    c_bits: int = 4
    r_bits: int = 4
    page_size: int = 64

    @property
    def codes_c_bytes(self) -> int:          # per token
        return self.d_c * self.c_bits // 8

    @property
    def codes_r_bytes(self) -> int:
        return self.d_r * self.r_bits // 8

    @property
    def meta_c_bytes(self) -> int:
        return (self.d_c // qz.GROUP) * 4

    @property
    def meta_r_bytes(self) -> int:
        return (self.d_r // qz.GROUP) * 4

    @property
    def token_bytes(self) -> int:
        return self.codes_c_bytes + self.codes_r_bytes + self.meta_c_bytes + self.meta_r_bytes

    def region_offsets(self):
        """Byte offset of each region inside a page."""
        P = self.page_size
        off_cc = 0
        off_cr = off_cc + P * self.codes_c_bytes
        off_mc = off_cr + P * self.codes_r_bytes
        off_mr = off_mc + P * self.meta_c_bytes
        end = off_mr + P * self.meta_r_bytes
        return off_cc, off_cr, off_mc, off_mr, end

    @property
    def page_bytes(self) -> int:
        end = self.region_offsets()[-1]
        return (end + 255) // 256 * 256


BF16_TOKEN_CHANNELS = 576


def bf16_page_bytes(fmt: CacheFormat) -> int:
    """A BF16 page stores ``P`` rows of ``d_c + d_r`` bf16 values."""
    return fmt.page_size * (fmt.d_c + fmt.d_r) * 2


def _token_byte_ranges(fmt: CacheFormat, slot: int):
    page, off = divmod(int(slot), fmt.page_size)
    base = page * fmt.page_bytes
    cc, cr, mc, mr, _ = fmt.region_offsets()
    return (
        (base + cc + off * fmt.codes_c_bytes, fmt.codes_c_bytes),
        (base + cr + off * fmt.codes_r_bytes, fmt.codes_r_bytes),
        (base + mc + off * fmt.meta_c_bytes, fmt.meta_c_bytes),
        (base + mr + off * fmt.meta_r_bytes, fmt.meta_r_bytes),
    )


def _meta_bytes(scale16: np.ndarray, zero16: np.ndarray) -> np.ndarray:
    """Interleave (scale, zero) fp16 pairs and view them as little-endian bytes."""
    pairs = np.stack([np.asarray(scale16, np.float16), np.asarray(zero16, np.float16)], axis=-1)
    return pairs.reshape(pairs.shape[0], -1).astype('<f2').view(np.uint8)


def encode_tokens(fmt: CacheFormat, c_kv_bits: np.ndarray, k_rope_bits: np.ndarray):
    """Quantize and pack ``n`` tokens; returns the four per-token byte blocks."""
    c_kv_bits = np.asarray(c_kv_bits, np.uint16).reshape(-1, fmt.d_c)
    k_rope_bits = np.asarray(k_rope_bits, np.uint16).reshape(-1, fmt.d_r)
    pc, sc, zc = qz.quantize_token_path(c_kv_bits, fmt.c_bits)
    pr, sr, zr = qz.quantize_token_path(k_rope_bits, fmt.r_bits)
    return pc, pr, _meta_bytes(sc, zc), _meta_bytes(sr, zr)


def write_tokens(cache: np.ndarray, fmt: CacheFormat, slots, c_kv_bits, k_rope_bits) -> None:
    """Slot-mapped insertion of quantized tokens into a flat uint8 page array."""
    blocks = encode_tokens(fmt, c_kv_bits, k_rope_bits)
    for i, slot in enumerate(np.asarray(slots, np.int64).reshape(-1)):
        if slot < 0:
            continue
        for (start, size), blk in zip(_token_byte_ranges(fmt, slot), blocks):
            cache[start:start + size] = blk[i]


def token_bytes_at(cache: np.ndarray, fmt: CacheFormat, slot: int) -> bytes:
    """The stored bytes of one token (codes_c | codes_r | meta_c | meta_r)."""
    return b"".join(cache[s:s + n].tobytes() for s, n in _token_byte_ranges(fmt, slot))


def read_tokens(cache: np.ndarray, fmt: CacheFormat, slots):
    """Reconstruct fp32 content latents ``[n, d_c]`` and RoPE keys ``[n, d_r]``."""
    slots = np.asarray(slots, np.int64).reshape(-1)
    n = slots.size
    pc = np.empty((n, fmt.codes_c_bytes), np.uint8)
    pr = np.empty((n, fmt.codes_r_bytes), np.uint8)
    mc = np.empty((n, fmt.meta_c_bytes), np.uint8)
    mr = np.empty((n, fmt.meta_r_bytes), np.uint8)
    for i, slot in enumerate(slots):
        for (start, size), dst in zip(_token_byte_ranges(fmt, slot), (pc, pr, mc, mr)):
            dst[i] = cache[start:start + size]
    mc16 = mc.view('<f2').reshape(n, -1, 2)
    mr16 = mr.view('<f2').reshape(n, -1, 2)
    c_hat = qz.dequantize_token_path(pc, mc16[..., 0], mc16[..., 1], fmt.c_bits)
    kr_hat = qz.dequantize_token_path(pr, mr16[..., 0], mr16[..., 1], fmt.r_bits)
    return c_hat, kr_hat


def encode_sequence_dense(fmt: CacheFormat, c_kv_bits, k_rope_bits):
    """Quantize then dequantize a whole sequence without paging (same arithmetic).

    Used where the oracle needs the reconstructed cache of many tokens at once:
    the values equal :func:`read_tokens` after :func:`write_tokens`.
    """
    c_kv_bits = np.asarray(c_kv_bits, np.uint16).reshape(-1, fmt.d_c)
    k_rope_bits = np.asarray(k_rope_bits, np.uint16).reshape(-1, fmt.d_r)
    pc, sc, zc = qz.quantize_token_path(c_kv_bits, fmt.c_bits)
    pr, sr, zr = qz.quantize_token_path(k_rope_bits, fmt.r_bits)
    c_hat = qz.dequantize_token_path(pc, sc, zc, fmt.c_bits)
    kr_hat = qz.dequantize_token_path(pr, sr, zr, fmt.r_bits)
    return c_hat, kr_hat

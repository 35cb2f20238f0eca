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

The paper's own storage (``meta="paper"``; Appendix C.4 last sentence,
Appendix C.5 "Storage layout"; reading 22 in the design doc) keeps three regions::

    codes_c[P][d_c * c_bits / 8]
    codes_r[P][d_r * r_bits / 8]
    meta   [P][32]   per token: bf16 content scales [d_c/64], byte content
                     zero-points [d_c/64], fp32 RoPE scales [d_r/64], byte
                     RoPE zero-points [d_r/64], zero padding to 32 bytes

which is 320 B per token and 20 480 B per 64-token page with 4-bit content,
the paper's figures (192 B and 12 288 B with 2-bit content).

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
    meta: str = "fp16"                      # or "paper"

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
    def paper_meta_bytes(self) -> int:       # per token, paper storage
        gc, gr = self.d_c // qz.GROUP, self.d_r // qz.GROUP
        return (3 * gc + 5 * gr + 15) // 16 * 16

    def region_sizes(self):
        """Bytes per token of each page region, in page order."""
        if self.meta == "paper":
            return [self.codes_c_bytes, self.codes_r_bytes, self.paper_meta_bytes]
        return [self.codes_c_bytes, self.codes_r_bytes, self.meta_c_bytes, self.meta_r_bytes]

    @property
    def token_bytes(self) -> int:
        return sum(self.region_sizes())

    def region_offsets(self):
        """Byte offset of each region inside a page, then the end of the last."""
        offs = [0]
        for n in self.region_sizes():
            offs.append(offs[-1] + self.page_size * n)
        return tuple(offs)

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
    return tuple((base + o + off * n, n) for o, n in zip(fmt.region_offsets()[:-1], fmt.region_sizes()))


def _meta_bytes(scale16: np.ndarray, zero16: np.ndarray) -> np.ndarray:
    """Interleave (scale, zero) fp16 pairs and view them as little-endian bytes."""
    pairs = np.stack([np.asarray(scale16, np.float16), np.asarray(zero16, np.float16)], axis=-1)
    return pairs.reshape(pairs.shape[0], -1).astype('<f2').view(np.uint8)


def _paper_meta_bytes(fmt: CacheFormat, sc, zc, sr, zr) -> np.ndarray:
    """The paper-storage metadata record of every token (layout above)."""
    n = sc.shape[0]
    rec = np.zeros((n, fmt.paper_meta_bytes), np.uint8)
    gc, gr = sc.shape[1], sr.shape[1]
    bf16_bits = (np.asarray(sc, np.float32).view(np.uint32) >> np.uint32(16)).astype('<u2')
    rec[:, 0:2 * gc] = bf16_bits.view(np.uint8).reshape(n, 2 * gc)
    rec[:, 2 * gc:3 * gc] = np.asarray(zc, np.uint8)
    rec[:, 3 * gc:3 * gc + 4 * gr] = np.asarray(sr, '<f4').view(np.uint8).reshape(n, 4 * gr)
    rec[:, 3 * gc + 4 * gr:3 * gc + 5 * gr] = np.asarray(zr, np.uint8)
    return rec


def _stored_meta(fmt: CacheFormat, c_kv_bits, k_rope_bits):
    c_kv_bits = np.asarray(c_kv_bits, np.uint16).reshape(-1, fmt.d_c)
    k_rope_bits = np.asarray(k_rope_bits, np.uint16).reshape(-1, fmt.d_r)
    pc, sc, zc = qz.quantize_token_path(c_kv_bits, fmt.c_bits, fmt.meta, rope=False)
    pr, sr, zr = qz.quantize_token_path(k_rope_bits, fmt.r_bits, fmt.meta, rope=True)
    return pc, sc, zc, pr, sr, zr


def encode_tokens(fmt: CacheFormat, c_kv_bits: np.ndarray, k_rope_bits: np.ndarray):
    """Quantize and pack ``n`` tokens; returns the per-token byte block of
    every page region."""
    pc, sc, zc, pr, sr, zr = _stored_meta(fmt, c_kv_bits, k_rope_bits)
    if fmt.meta == "paper":
        return pc, pr, _paper_meta_bytes(fmt, sc, zc, sr, zr)
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
    blocks = [np.empty((n, size), np.uint8) for size in fmt.region_sizes()]
    for i, slot in enumerate(slots):
        for (start, size), dst in zip(_token_byte_ranges(fmt, slot), blocks):
            dst[i] = cache[start:start + size]
    return decode_blocks(fmt, blocks)


def page_blocks(fmt: CacheFormat, pages: np.ndarray, n: int):
    """The per-token byte blocks of every region (page order) of the first
    ``n`` tokens stored in consecutive pages ``pages [num, page_bytes]``
    (token ``t`` at page ``t // P``, offset ``t % P``)."""
    pages = np.asarray(pages, np.uint8).reshape(-1, fmt.page_bytes)
    offs = fmt.region_offsets()
    out = []
    for o, size in zip(offs[:-1], fmt.region_sizes()):
        reg = pages[:, o:o + fmt.page_size * size].reshape(-1, size)
        out.append(np.ascontiguousarray(reg[:n]))
    return out


def decode_blocks(fmt: CacheFormat, blocks):
    """Reconstruct fp32 ``(c_hat [n, d_c], kr_hat [n, d_r])`` from the per-token
    region blocks of :func:`encode_tokens` / :func:`page_blocks`."""
    n = blocks[0].shape[0]
    pc, pr = blocks[0], blocks[1]
    if fmt.meta == "paper":
        rec = blocks[2]
        gc, gr = fmt.d_c // qz.GROUP, fmt.d_r // qz.GROUP
        sc = qz.bf16_bits_to_f32(np.ascontiguousarray(rec[:, 0:2 * gc]).view('<u2'))
        zc = rec[:, 2 * gc:3 * gc]
        sr = np.ascontiguousarray(rec[:, 3 * gc:3 * gc + 4 * gr]).view('<f4')
        zr = rec[:, 3 * gc + 4 * gr:3 * gc + 5 * gr]
    else:
        mc16 = blocks[2].view('<f2').reshape(n, -1, 2)
        mr16 = blocks[3].view('<f2').reshape(n, -1, 2)
        sc, zc, sr, zr = mc16[..., 0], mc16[..., 1], mr16[..., 0], mr16[..., 1]
    c_hat = qz.dequantize_token_path(pc, sc, zc, fmt.c_bits)
    kr_hat = qz.dequantize_token_path(pr, sr, zr, fmt.r_bits)
    return c_hat, kr_hat


def encode_sequence_dense(fmt: CacheFormat, c_kv_bits, k_rope_bits):
    """Quantize then dequantize a whole sequence without paging (same arithmetic).

    Used where the oracle needs the reconstructed cache of many tokens at once:
    the values equal :func:`read_tokens` after :func:`write_tokens`.
    """
    pc, sc, zc, pr, sr, zr = _stored_meta(fmt, c_kv_bits, k_rope_bits)
    c_hat = qz.dequantize_token_path(pc, sc, zc, fmt.c_bits)
    kr_hat = qz.dequantize_token_path(pr, sr, zr, fmt.r_bits)
    return c_hat, kr_hat

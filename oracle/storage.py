"""Per-layer persistent storage accounting -- oracle (test infrastructure).

Appendix C.5, "Storage layout" and eq. physical_cache_storage: for a request
of ``L`` tokens and 64-token pages, the paper's packed C4R4 layout costs
``ceil(L/64) * (20480 + 8) + 152064`` bytes (packed pages, an 8-byte reverse
page mapping per page, and 132 protected BF16 tokens of 576 channels), while a
BF16 cache costs ``ceil(L/64) * 73728`` bytes.  The paper prints the ratios
3.22x at 4K and 3.59x at 128K.

The library's own layout (fp16 scale and fp16 zero for every group) is also
accounted here, so its packed-only compression against BF16 can be reported.
"""
from __future__ import annotations

import math

PAPER_C4R4_PAGE = 20480      # bytes per 64-token page, paper layout
REVERSE_MAP = 8              # bytes per physical page
PROTECTION = 132 * 576 * 2   # sink 4 + recent 128 BF16 tokens per request and layer
BF16_PAGE = 64 * 1152


def paper_c4r4_bytes(L: int) -> int:
    return math.ceil(L / 64) * (PAPER_C4R4_PAGE + REVERSE_MAP) + PROTECTION


def bf16_bytes(L: int) -> int:
    return math.ceil(L / 64) * BF16_PAGE


def paper_compression(L: int) -> float:
    return bf16_bytes(L) / paper_c4r4_bytes(L)


def packed_token_bytes(d_c: int, d_r: int, c_bits: int, r_bits: int, group: int = 64,
                       meta_bytes_per_group: int = 4) -> int:
    """Codes plus per-group metadata of one token in the library layout."""
    return (d_c * c_bits + d_r * r_bits) // 8 + (d_c // group + d_r // group) * meta_bytes_per_group


def packed_compression(d_c: int = 512, d_r: int = 64, c_bits: int = 4, r_bits: int = 4) -> float:
    """Packed-only compression of the library layout against a BF16 cache."""
    return (d_c + d_r) * 2 / packed_token_bytes(d_c, d_r, c_bits, r_bits)

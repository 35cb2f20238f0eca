"""Pins for the paper's own cache storage in the oracle (CPU only).

Appendix C.4 (last sentence) stores content scales in BF16 and RoPE scales in
FP32; Appendix C.5 ("Storage layout", eq. physical_cache_storage) prints
20 480 B per 64-token C4R4 page (320 B per token) and the 3.22x / 3.59x
storage ratios against a BF16 cache.  Checked here: the page geometry against
those printed numbers, the bf16 rounding of scales against brute-force
nearest-even search, a hand-built metadata record byte by byte, the
quantization error bound with a rounded scale, the exact fp32 RoPE scale, and
the write/read round trip.
"""
import math

import numpy as np
import pytest

from oracle import paged_cache as pc
from oracle import quantizer as qz
from oracle import storage

PAPER = pc.CacheFormat(meta="paper")


def test_page_geometry_matches_the_printed_numbers():
    assert PAPER.token_bytes == 320
    assert PAPER.page_bytes == 20480 == storage.PAPER_C4R4_PAGE
    assert PAPER.region_offsets() == (0, 16384, 18432, 20480)
    c2 = pc.CacheFormat(c_bits=2, meta="paper")
    assert c2.token_bytes == 192 and c2.page_bytes == 12288
    # eq. physical_cache_storage with this layout's page size: the printed ratios
    for L, ratio in ((4096, 3.22), (131072, 3.59)):
        m_c4r4 = math.ceil(L / 64) * (PAPER.page_bytes + 8) + 132 * 576 * 2
        m_bf16 = math.ceil(L / 64) * pc.bf16_page_bytes(PAPER)
        assert round(m_bf16 / m_c4r4, 2) == ratio


def _nearest_even_bf16(x: float) -> float:
    """Brute force: the bf16 neighbours of x, nearest, ties to an even mantissa."""
    b = int(np.float32(x).view(np.uint32))
    lo = b & 0xFFFF0000
    hi = lo + 0x10000
    cands = [lo, hi]
    xv = float(np.float32(x))
    vals = [float(np.uint32(c).view(np.float32)) for c in cands]
    d = [abs(v - xv) for v in vals]
    if d[0] != d[1]:
        return vals[int(d[1] < d[0])]
    return vals[0] if ((lo >> 16) & 1) == 0 else vals[1]


def test_bf16_rounding_is_nearest_even():
    rng = np.random.default_rng(0)
    xs = (rng.standard_normal(4000) * 10.0 ** rng.uniform(-12, 6, 4000)).astype(np.float32)
    # exact ties: the low 16 bits are 0x8000, with both mantissa parities
    ties = (rng.integers(0x3000, 0x4800, 200).astype(np.uint32) << 16 | 0x8000).view(np.float32)
    for x in np.concatenate([xs, ties, -ties]):
        assert qz.f32_to_bf16(np.float32(x)) == np.float32(_nearest_even_bf16(float(x)))


def _bits(x):
    b = np.ascontiguousarray(x, np.float32).view(np.uint32)
    assert np.all(b & 0xFFFF == 0)
    return (b >> 16).astype(np.uint16)


def test_hand_built_metadata_record():
    """Content group 3 spans [-1, 14] (s = 1, z = 1); the other content groups
    are all zero; the RoPE group spans [0.5, 2] (s = 0.1 in fp32, z = 0)."""
    c = np.zeros((1, 512), np.float32)
    c[0, 192:256] = 0.0
    c[0, 192] = -1.0
    c[0, 193] = 14.0
    r = np.full((1, 64), 1.0, np.float32)
    r[0, 0] = 0.5
    r[0, 1] = 2.0
    pcodes, pr, rec = pc.encode_tokens(PAPER, _bits(c), _bits(r))
    rec = rec[0]
    assert rec.shape == (32,)
    assert bytes(rec[6:8]) == b"\x80\x3f"                        # bf16(1.0)
    assert rec[16 + 3] == 1 and all(rec[16 + g] == 0 for g in range(8) if g != 3)
    assert bytes(rec[24:28]) == np.float32(1.5 / 15).tobytes()   # fp32 scale, not rounded further
    assert rec[28] == 0 and not rec[29:].any()
    # an all-zero group stores bf16(1e-8 / 15) and zero-point 0
    eps_scale = qz.f32_to_bf16(np.float32(1e-8) / np.float32(15))
    assert bytes(rec[0:2]) == (np.asarray(eps_scale, np.float32).view(np.uint32) >> 16).astype('<u2').tobytes()
    # codes of group 3: -1 -> 0, 14 -> 15, 0 -> 1
    q = qz.unpack_codes(pcodes, 4)[0, 192:256]
    assert q[0] == 0 and q[1] == 15 and np.all(q[2:] == 1)


@pytest.mark.parametrize("c_bits", [4, 2])
def test_error_bound_with_rounded_scales(c_bits):
    """|x - s_b (q - z)| <= s/2 + m |s - s_b| inside the clip range, with
    |s - s_b| <= 2^-8 s for the bf16 content scale (nearest rounding to 8
    significant bits)."""
    rng = np.random.default_rng(c_bits)
    x = (rng.standard_normal((300, 512)) * 10.0 ** rng.uniform(-3, 3, (300, 1))).astype(np.float32)
    xb = _bits(qz.f32_to_bf16(x))
    x64 = qz.bf16_bits_to_f32(xb).astype(np.float64).reshape(300, 8, 64)
    q, s, z = qz.quantize_groups(x64.astype(np.float32), c_bits)
    packed, sb, zb = qz.quantize_token_path(xb, c_bits, "paper", rope=False)
    assert np.all(np.abs(s - sb) <= 2.0 ** -8 * s)
    xh = qz.dequantize_token_path(packed, sb, zb, c_bits).astype(np.float64).reshape(300, 8, 64)
    m = (1 << c_bits) - 1
    lo = -z[..., None] * s[..., None]
    hi = (m - z[..., None]) * s[..., None]
    inside = (x64 >= lo) & (x64 <= hi)
    bound = s[..., None] / 2 * (1 + 1e-5) + m * np.abs(s - sb)[..., None] + 1e-30
    assert np.all(np.abs(x64 - xh)[inside] <= np.broadcast_to(bound, x64.shape)[inside])


def test_rope_path_dequantizes_with_the_exact_fp32_scale():
    rng = np.random.default_rng(3)
    k = _bits(qz.f32_to_bf16(rng.standard_normal((50, 64)).astype(np.float32)))
    packed, sr, zr = qz.quantize_token_path(k, 4, "paper", rope=True)
    q, s, z = qz.quantize_groups(qz.bf16_bits_to_f32(k).reshape(50, 1, 64), 4)
    assert np.array_equal(sr, s)
    want = (s[..., None] * (q.astype(np.float32) - z[..., None])).astype(np.float32).reshape(50, 64)
    assert np.array_equal(qz.dequantize_token_path(packed, sr, zr, 4), want)


@pytest.mark.parametrize("c_bits", [4, 2])
def test_write_read_round_trip(c_bits):
    f = pc.CacheFormat(c_bits=c_bits, meta="paper")
    rng = np.random.default_rng(10 + c_bits)
    n = 70
    c = _bits(qz.f32_to_bf16((rng.standard_normal((n, 512)) * 3).astype(np.float32)))
    k = _bits(qz.f32_to_bf16(rng.standard_normal((n, 64)).astype(np.float32)))
    cache = np.full(3 * f.page_bytes, 0xA5, np.uint8)
    slots = rng.permutation(3 * 64)[:n]
    pc.write_tokens(cache, f, slots, c, k)
    ch, kh = pc.read_tokens(cache, f, slots)
    dc, dk = pc.encode_sequence_dense(f, c, k)
    assert np.array_equal(ch, dc) and np.array_equal(kh, dk)
    # the fp16-metadata layout reconstructs differently (other stored scales)
    fc, fk = pc.encode_sequence_dense(pc.CacheFormat(c_bits=c_bits), c, k)
    assert not np.array_equal(fc, dc)

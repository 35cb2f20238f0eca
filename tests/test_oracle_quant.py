"""Pins for the quantizer/packing/page-layout oracle (CPU only).

Each check is fixed by something outside the oracle's own code: hand-derived
cases of the Appendix C.4 quantizer (tests/golden/quant_hand_cases.json), the
bound a round-to-nearest quantizer must meet, exhaustive pack/unpack round
trips, the byte offsets the page layout defines, and the storage ratios the
paper prints (Appendix C.5, eq. physical_cache_storage).
"""
import json
import os

import numpy as np
import pytest

from oracle import paged_cache as pc
from oracle import quantizer as qz
from oracle import storage

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quant_hand_cases.json")


def _cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def _group(case):
    g = np.full(64, case["fill"], dtype=np.float32)
    g[:len(case["head"])] = case["head"]
    return g


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_hand_cases(case):
    bits = case["bits"]
    g = _group(case)
    q, s, z = qz.quantize_groups(g[None], bits)
    assert format(int(np.float32(s[0]).view(np.uint32)), "08x") == case["s_f32_hex"]
    assert int(z[0]) == case["z"]
    n = len(case["head"])
    assert q[0, :n].tolist() == case["q_head"]
    assert np.all(q[0, n:] == case["q_fill"])
    packed = qz.pack_codes(q, bits)[0]
    want = bytes.fromhex(case["packed_head_hex"])
    assert packed[:len(want)].tobytes() == want
    s16, z16 = qz.stored_meta(s, z)
    assert format(int(s16.view(np.uint16)[0]), "04x") == case["scale_f16_hex"]
    assert format(int(z16.view(np.uint16)[0]), "04x") == case["zero_f16_hex"]
    xh = qz.dequantize(q, s16, z16)[0]
    np.testing.assert_allclose(xh[:n], np.float32(case["xhat_head"]), rtol=1e-7, atol=0)
    np.testing.assert_allclose(xh[n:], np.float32(case["xhat_fill"]), rtol=1e-7, atol=0)
    if "xhat_fill_signbit" in case:
        assert np.all(np.signbit(xh[n:]) == bool(case["xhat_fill_signbit"]))


@pytest.mark.parametrize("bits", [2, 4])
def test_pack_unpack_all_bytes(bits):
    # every byte value in every byte position of a word, and random words
    every = np.zeros((4, 256, 4), np.uint8)
    for pos in range(4):
        every[pos, :, pos] = np.arange(256)
    rnd = np.random.default_rng(3).integers(0, 256, (512, 4), dtype=np.uint8)
    packed = np.concatenate([every.reshape(1024, 4), rnd]).reshape(1, -1)
    codes = qz.unpack_codes(packed, bits)
    assert codes.shape == (1, packed.shape[1] * 8 // bits)
    assert codes.max() == (1 << bits) - 1
    assert np.array_equal(qz.pack_codes(codes, bits), packed)
    # field order, written out per byte: byte 0 of a word holds the even
    # channels 0, 2, .. (lowest bits first), byte 2 the odd channels 1, 3, ..
    per = 32 // bits
    words = codes.reshape(-1, per)
    mask = (1 << bits) - 1
    b = packed.reshape(-1, 4)
    for k in range(8 // bits):
        assert np.array_equal(words[:, 2 * k], (b[:, 0] >> (bits * k)) & mask)
        assert np.array_equal(words[:, 2 * k + 1], (b[:, 2] >> (bits * k)) & mask)
        assert np.array_equal(words[:, 2 * (k + 8 // bits)], (b[:, 1] >> (bits * k)) & mask)
        assert np.array_equal(words[:, 2 * (k + 8 // bits) + 1], (b[:, 3] >> (bits * k)) & mask)


@pytest.mark.parametrize("bits", [2, 4])
def test_round_to_nearest_bound(bits):
    rng = np.random.default_rng(7)
    x = rng.standard_normal((20000, 64)).astype(np.float32) * rng.uniform(0.01, 20, (20000, 1)).astype(np.float32)
    x += rng.uniform(-0.2, 0.2, (20000, 1)).astype(np.float32)
    q, s, z = qz.quantize_groups(x, bits)
    m = (1 << bits) - 1
    assert q.max() <= m and z.min() >= 0 and z.max() <= m
    straddle = (x.min(1) <= s / 2) & (x.max(1) >= -s / 2)
    assert straddle.mean() > 0.9
    xs, ss, qs, zs = x[straddle], s[straddle, None], q[straddle], z[straddle, None]
    err = np.abs(xs.astype(np.float64) - ss.astype(np.float64) * (qs.astype(np.float64) - zs))
    # half a step, plus the two fp32 roundings of x/s + z before rint
    slack = ss.astype(np.float64) * (np.abs(xs / ss) + zs) * 2.0 ** -23
    assert np.all(err <= ss / 2 + slack)
    # with the stored fp16 scale: half a step plus m times the scale rounding
    s16, z16 = qz.stored_meta(s, z)
    xh = qz.dequantize(q, s16, z16)[straddle].astype(np.float64)
    bound = ss / 2 + m * np.abs(ss.astype(np.float64) - s16[straddle, None].astype(np.float64)) + slack
    assert np.all(np.abs(xs - xh) <= bound * (1 + 2.0 ** -20))


def test_fp16_subnormal_scale_round_trip():
    rng = np.random.default_rng(3)
    x = (rng.uniform(-1, 1, (64, 64)) * 5e-5).astype(np.float32)
    q, s, z = qz.quantize_groups(x, 4)
    s16, _ = qz.stored_meta(s, z)
    f = s16.astype(np.float32)
    assert np.all((f > 0) & (f < np.float32(6.103515625e-05)))       # fp16 subnormal range
    # round-half-to-even to the nearest multiple of 2**-24
    k = s.astype(np.float64) / 2.0 ** -24
    lo = np.floor(k)
    near = np.where(k - lo > 0.5, lo + 1, np.where(k - lo < 0.5, lo, lo + (lo % 2)))
    assert np.array_equal(f.astype(np.float64), near * 2.0 ** -24)


def test_dequant_zero_code_is_zero():
    q = np.arange(16, dtype=np.uint8)[None, None, :].repeat(4, 2)[..., :64]
    s16 = np.float16([[0.37]])
    for zv in range(16):
        z16 = np.float16([[zv]])
        xh = qz.dequantize(q, s16, z16)
        assert np.all(xh[q == zv] == 0)
        assert np.all(np.sign(xh[q != zv]) == np.sign(q[q != zv].astype(int) - zv))


@pytest.mark.parametrize("c_bits,page,token,offs", [
    (4, 20736, 324, (0, 16384, 18432, 20480, 20736)),
    (2, 12544, 196, (0, 8192, 10240, 12288, 12544)),
])
def test_page_layout_offsets(c_bits, page, token, offs):
    f = pc.CacheFormat(c_bits=c_bits)
    assert f.page_bytes == page and f.token_bytes == token
    assert f.region_offsets() == offs
    assert f.page_bytes % 256 == 0
    assert pc.bf16_page_bytes(f) == 73728


def test_page_write_places_hand_case_bytes():
    """Hand case A in content group 1 of token 5 of page 2 lands at the computed bytes."""
    f = pc.CacheFormat(c_bits=4)
    case = _cases()[0]
    c = np.zeros((1, 512), np.float32)
    c[0, 64:128] = _group(case)
    kr = np.zeros((1, 64), np.float32)
    kr[0, :2] = [-1.0, 2.0]                                     # hand case D in the RoPE group
    to_bits = lambda a: (a.view(np.uint32) >> 16).astype(np.uint16)   # exact: values are bf16
    cache = np.zeros(3 * f.page_bytes, np.uint8)
    slot = 2 * 64 + 5
    pc.write_tokens(cache, f, [slot, -1], np.vstack([to_bits(c), to_bits(c)]), np.vstack([to_bits(kr), to_bits(kr)]))
    base = 2 * f.page_bytes
    codes = cache[base + 5 * 256: base + 6 * 256]
    assert codes[32:37].tobytes() == bytes.fromhex("806a8f7677")
    rope = cache[base + 16384 + 5 * 32: base + 16384 + 6 * 32]
    assert rope[:4].tobytes() == bytes.fromhex("50555f55")
    meta_c = cache[base + 18432 + 5 * 32: base + 18432 + 6 * 32].view("<u2")
    assert meta_c[2] == 0x3C00 and meta_c[3] == 0x4700            # group 1: scale 1, zero 7
    meta_r = cache[base + 20480 + 5 * 4: base + 20480 + 6 * 4].view("<u2")
    assert meta_r[0] == 0x3266 and meta_r[1] == 0x4500
    assert np.count_nonzero(cache[:base]) == 0                    # the skipped token wrote nothing
    c_hat, kr_hat = pc.read_tokens(cache, f, [slot])
    assert c_hat[0, 64:72].tolist() == [-7, 8, 1, 1, 3, -1, -1, 0]
    np.testing.assert_allclose(kr_hat[0, :2], [-0.99975586, 1.9995117], rtol=1e-7)


def test_dense_encode_matches_paged_read():
    rng = np.random.default_rng(11)
    for c_bits in (2, 4):
        f = pc.CacheFormat(c_bits=c_bits)
        n = 70
        c = (rng.standard_normal((n, 512)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        k = (rng.standard_normal((n, 64)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        cache = np.zeros(2 * f.page_bytes, np.uint8)
        slots = np.arange(n)[::-1]
        pc.write_tokens(cache, f, slots, c, k)
        ch, kh = pc.read_tokens(cache, f, slots)
        dc, dk = pc.encode_sequence_dense(f, c, k)
        assert np.array_equal(ch, dc) and np.array_equal(kh, dk)


def test_storage_ratios_printed_by_paper():
    # Appendix C.5: "3.22x at 4K and 3.59x at 128K"
    assert round(storage.paper_compression(4096), 2) == 3.22
    assert round(storage.paper_compression(131072), 2) == 3.59
    assert storage.paper_c4r4_bytes(64) == 20480 + 8 + 152064
    assert storage.packed_token_bytes(512, 64, 4, 4) == 324
    assert storage.packed_token_bytes(512, 64, 2, 4) == 196
    assert abs(storage.packed_compression(c_bits=4) - 1152 / 324) < 1e-12

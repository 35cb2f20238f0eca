"""GPU parity of the writers: packed codes and fp16 metadata bit-exact.

The GPU quantize-append must produce the same cache bytes as the oracle's
quantizer and page layout (Appendix C.4; Appendix C.5), with fp16 metadata
and with the paper's bf16 / fp32 scales, for every token: the
hand-derived cases, random tokens with outlier channels over 12 decades of
scale, constant groups, fp16-subnormal scales, signed zeros, skipped slots.
Bytes the writer must not touch are checked too (both caches start from the
same fill pattern).
"""
import json
import os

import numpy as np
import pytest

from oracle import paged_cache as pc

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quant_hand_cases.json")


def _bits(x):
    b = np.ascontiguousarray(x, np.float32).view(np.uint32)
    assert np.all(b & 0xFFFF == 0), "test values must be exactly representable in bf16"
    return (b >> 16).astype(np.uint16)


def _round_bf16(x):
    b = np.ascontiguousarray(x, np.float32).view(np.uint32)
    return (((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16).astype(np.uint32).view(np.float32)


def _tokens(c_bits, rng):
    cases = json.load(open(GOLDEN))["cases"]
    groups4 = []
    groups_c = []
    for c in cases:
        g = np.full(64, c["fill"], np.float32)
        g[:len(c["head"])] = c["head"]
        if c["bits"] == 4:
            groups4.append(g)
        if c["bits"] == c_bits:
            groups_c.append(g)
    rows_c, rows_r = [], []
    # hand cases: content group (i % 8) and the RoPE group of token i
    for i in range(max(len(groups_c), len(groups4))):
        c = rng.standard_normal(512).astype(np.float32)
        c[64 * (i % 8):64 * (i % 8) + 64] = groups_c[i % len(groups_c)]
        rows_c.append(c)
        rows_r.append(groups4[i % len(groups4)])
    # random tokens: outlier channels, per-token scale over 12 decades
    n = 600
    c = rng.standard_normal((n, 512)).astype(np.float32)
    c[:, rng.choice(512, 6, replace=False)] *= 10
    c *= 10.0 ** rng.uniform(-6, 6, (n, 1)).astype(np.float32)
    r = rng.standard_normal((n, 64)).astype(np.float32) * 10.0 ** rng.uniform(-6, 6, (n, 1)).astype(np.float32)
    rows_c.extend(c)
    rows_r.extend(r)
    # special groups
    special = [np.full(64, 0.0), np.full(64, -0.0), np.full(64, 3.0), np.full(64, -1e30),
               np.linspace(-1e-4, 1e-4, 64), np.linspace(2e-5, 9e-5, 64),   # fp16-subnormal scales
               np.where(np.arange(64) % 2 == 0, 1e38, -1e38), np.linspace(1000, 1001, 64)]
    for i, g in enumerate(special):
        cc = np.tile(np.asarray(g, np.float32), 8)
        rows_c.append(cc)
        rows_r.append(np.asarray(special[(i + 3) % len(special)], np.float32))
    C = _round_bf16(np.stack(rows_c))
    R = _round_bf16(np.stack(rows_r))
    return _bits(C), _bits(R)


@pytest.mark.parametrize("meta", ["fp16", "paper"])
@pytest.mark.parametrize("c_bits", [4, 2])
def test_quant_append_bit_exact(c_bits, meta):
    import torch

    from paper_2609_36760_amd import _binding as mb
    rng = np.random.default_rng(100 + c_bits)
    cb, rb = _tokens(c_bits, rng)
    n = cb.shape[0]
    fmt = pc.CacheFormat(c_bits=c_bits, meta=meta)
    mfmt = mb.cache_format(c_bits=c_bits, meta=mb.MLA_META_PAPER if meta == "paper" else mb.MLA_META_FP16)
    num_pages = (n + 40) // 64 + 3
    num_slots = num_pages * 64
    slots = rng.permutation(num_slots)[:n].astype(np.int64)
    slots[5] = -1                       # skipped
    slots[17] = num_slots + 7           # beyond the cache: skipped
    assert fmt.page_bytes == mb.mla_lowbit_page_bytes(mfmt)
    want = np.full(num_pages * fmt.page_bytes, 0x5A, np.uint8)
    keep = slots.copy()
    keep[keep >= num_slots] = -1
    pc.write_tokens(want, fmt, keep, cb, rb)

    dev = "cuda"
    cache = torch.full((num_pages * fmt.page_bytes,), 0x5A, dtype=torch.uint8, device=dev)
    mb.mla_lowbit_quant_append(mfmt, torch.from_numpy(cb.view(np.int16)).to(dev),
                               torch.from_numpy(rb.view(np.int16)).to(dev), torch.from_numpy(slots).to(dev),
                               cache, num_pages)
    got = cache.cpu().numpy()
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} bytes differ, first at {bad[:8]}"


def test_quant_append_strided_rows():
    """c_kv and k_rope as column slices of one [n, 576] buffer (row stride 576)."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    rng = np.random.default_rng(7)
    n = 130
    full = _bits(_round_bf16(rng.standard_normal((n, 576)).astype(np.float32)))
    fmt = pc.CacheFormat(c_bits=4)
    want = np.zeros(3 * fmt.page_bytes, np.uint8)
    slots = np.arange(n, dtype=np.int64)[::-1].copy()
    pc.write_tokens(want, fmt, slots, full[:, :512], full[:, 512:])
    t = torch.from_numpy(full.view(np.int16)).cuda()
    cache = torch.zeros(3 * fmt.page_bytes, dtype=torch.uint8, device="cuda")
    mb.mla_lowbit_quant_append(mb.cache_format(c_bits=4), t[:, :512], t[:, 512:],
                               torch.from_numpy(slots).cuda(), cache, 3)
    assert np.array_equal(cache.cpu().numpy(), want)


def test_bf16_append_copies_rows():
    import torch

    from paper_2609_36760_amd import _binding as mb
    rng = np.random.default_rng(8)
    n = 100
    c = rng.integers(0, 1 << 16, (n, 512), dtype=np.uint16)
    k = rng.integers(0, 1 << 16, (n, 64), dtype=np.uint16)
    slots = rng.permutation(192)[:n].astype(np.int64)
    slots[3] = -1
    cache = torch.zeros(3 * 73728, dtype=torch.uint8, device="cuda")
    mb.mla_bf16_append(mb.cache_format(), torch.from_numpy(c.view(np.int16)).cuda(),
                       torch.from_numpy(k.view(np.int16)).cuda(), torch.from_numpy(slots).cuda(), cache, 3)
    got = cache.cpu().numpy().view(np.uint16).reshape(192, 576)
    want = np.zeros((192, 576), np.uint16)
    for i, s in enumerate(slots):
        if s >= 0:
            want[s, :512], want[s, 512:] = c[i], k[i]
    assert np.array_equal(got, want)


def test_empty_append_is_noop():
    import torch

    from paper_2609_36760_amd import _binding as mb
    cache = torch.zeros(20736, dtype=torch.uint8, device="cuda")
    e = torch.zeros((0, 512), dtype=torch.int16, device="cuda")
    mb.mla_lowbit_quant_append(mb.cache_format(), e, e[:, :64], torch.zeros(0, dtype=torch.int64, device="cuda"),
                               cache, 1)
    torch.cuda.synchronize()
    assert int(cache.count_nonzero()) == 0

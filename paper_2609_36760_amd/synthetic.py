"""Seeded synthetic inputs for low-bit MLA decode workloads.

This module only draws random inputs and page tables; it contains none of the
attention or quantization arithmetic.  Both the GPU library's tests/benchmark
and the CPU oracle consume what it produces.

Recipe (DeepSeek-V3-class MLA shapes: latent 512, RoPE key 64):
  * every stream is numpy ``PCG64`` seeded by ``SeedSequence(1000*cfg + k,
    spawn_key=(layer, b))`` so any single sequence can be regenerated alone;
    ``k``: 0 outlier channels, 1 content latent, 2 RoPE key, 3 content query,
    4 RoPE query, 5 sequence lengths, 6 physical page permutation;
  * content latent ``c_kv ~ N(0, 1)``; a fixed, seeded subset of channels
    (``round(frac * 512)``) is multiplied by an outlier factor;
  * RoPE key: frequency pair ``i`` (channels ``2i, 2i+1``) draws
    ``N(0, sigma_i^2)`` with ``sigma_i = 0.1 * 50**(i/31)`` (log-spaced
    0.1..5), then is rotated by ``t * 10000**(-2i/64)`` for token position ``t``;
  * queries ``q_lat, q_rope ~ N(0, 1)``;
  * every value is rounded to bf16 (round-half-to-even) and handled as its
    uint16 bit pattern;
  * physical pages are a seeded permutation, so no sequence owns a contiguous
    range of pages;
  * contexts too long for the host (the 16-head grid up to 1M tokens) draw the
    same distributions on the GPU from a seeded torch generator
    (:func:`device_sequence_tokens`).
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

D_C = 512
D_R = 64
PAGE = 64


@dataclass(frozen=True)
class Workload:
    name: str
    cfg: int                      # seed namespace
    B: int
    H: int
    s_q: int
    context: int | None           # uniform context length (tokens incl. queries), or None
    layers: tuple = ((4, 4),)     # (content bits, RoPE bits) per layer
    outlier_frac: float = 0.01
    outlier_mult: float = 10.0
    split_tokens: int = 0
    ctx_range: tuple | None = None  # (lo, hi) for log-uniform ragged lengths
    description: str = field(default="", compare=False)

    @property
    def tau(self) -> float:
        return 1.0 / math.sqrt(192.0)


WORKLOADS = {
    "tiny_b1_h16_256": Workload(
        "tiny_b1_h16_256", 0, B=1, H=16, s_q=1, context=256,
        description="batch 1, 16 heads, context 256, INT4 content + INT4 RoPE key"),
    "dsv3_b32_h128_4k_c4r4": Workload(
        "dsv3_b32_h128_4k_c4r4", 1, B=32, H=128, s_q=1, context=4096, split_tokens=512,
        description="batch 32, 128 heads, context 4096, INT4/INT4"),
    "int2_b64_h128_32k_c2r4": Workload(
        "int2_b64_h128_32k_c2r4", 2, B=64, H=128, s_q=1, context=32768, layers=((2, 4),),
        outlier_frac=0.02, outlier_mult=8.0, split_tokens=8192,
        description="batch 64, 128 heads, context 32768, INT2 content + INT4 RoPE key"),
    "splitkv_b8_h128_128k_c4r4": Workload(
        "splitkv_b8_h128_128k_c4r4", 3, B=8, H=128, s_q=1, context=131072, split_tokens=2048,
        description="batch 8, 128 heads, context 131072, INT4/INT4, 64 KV chunks"),
    "ragged_b96_h128_sq2_mixed": Workload(
        "ragged_b96_h128_sq2_mixed", 4, B=96, H=128, s_q=2, context=None, layers=((4, 4), (2, 4)),
        ctx_range=(1024, 131072), split_tokens=4096,
        description="96 ragged sequences (log-uniform 1K-128K), 2 causal queries, "
                    "one INT4/INT4 and one INT2/INT4 layer, 2 appended tokens each"),
    "c4r4_b64_h128_32k": Workload(
        "c4r4_b64_h128_32k", 5, B=64, H=128, s_q=1, context=32768, split_tokens=8192,
        description="batch 64, 128 heads, context 32768, INT4/INT4"),
}


def _rng(cfg: int, k: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(1000 * cfg + k, spawn_key=key)))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round-half-to-even); finite inputs only."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def outlier_channels(w: Workload) -> np.ndarray:
    n = int(round(w.outlier_frac * D_C))
    return np.sort(_rng(w.cfg, 0).choice(D_C, size=n, replace=False))


def seq_lens(w: Workload) -> np.ndarray:
    if w.context is not None:
        return np.full(w.B, w.context, dtype=np.int32)
    lo, hi = w.ctx_range
    u = _rng(w.cfg, 5).uniform(math.log(lo), math.log(hi), size=w.B)
    return np.floor(np.exp(u)).astype(np.int32)


def sequence_tokens(w: Workload, layer: int, b: int, L: int, start: int = 0):
    """bf16 bit patterns of tokens ``[start, L)`` of sequence ``b``.

    Returns ``(c_kv [L-start, 512], k_rope [L-start, 64])`` as uint16.  The
    stream is drawn from position 0, so any sub-range is consistent with the
    whole sequence.
    """
    g = _rng(w.cfg, 1, layer, b)
    c = g.standard_normal((L, D_C), dtype=np.float32)[start:]
    c[:, outlier_channels(w)] *= np.float32(w.outlier_mult)
    g = _rng(w.cfg, 2, layer, b)
    i = np.arange(D_R // 2, dtype=np.float64)
    sigma = 0.1 * 50.0 ** (i / 31.0)
    xy = g.standard_normal((L, D_R // 2, 2), dtype=np.float32)[start:].astype(np.float64)
    xy *= sigma[None, :, None]
    theta = 10000.0 ** (-2.0 * i / D_R)
    ang = np.arange(start, L, dtype=np.float64)[:, None] * theta[None, :]
    cs, sn = np.cos(ang), np.sin(ang)
    kr = np.empty((L - start, D_R), dtype=np.float32)
    kr[:, 0::2] = xy[..., 0] * cs - xy[..., 1] * sn
    kr[:, 1::2] = xy[..., 0] * sn + xy[..., 1] * cs
    return f32_to_bf16_bits(c), f32_to_bf16_bits(kr)


def queries(w: Workload, layer: int = 0, batch=None):
    """bf16 queries ``q_lat [B, s_q, H, 512]`` and ``q_rope [B, s_q, H, 64]``."""
    bs = range(w.B) if batch is None else batch
    ql = np.empty((len(bs), w.s_q, w.H, D_C), np.uint16)
    qr = np.empty((len(bs), w.s_q, w.H, D_R), np.uint16)
    for j, b in enumerate(bs):
        ql[j] = f32_to_bf16_bits(_rng(w.cfg, 3, layer, b).standard_normal((w.s_q, w.H, D_C), dtype=np.float32))
        qr[j] = f32_to_bf16_bits(_rng(w.cfg, 4, layer, b).standard_normal((w.s_q, w.H, D_R), dtype=np.float32))
    return ql, qr


def page_table(w: Workload, lens: np.ndarray, layer: int = 0, page: int = PAGE):
    """Seeded page permutation of ``page``-token pages:
    ``(block_table [B, max_pages] int32, num_pages)``.

    Unused table entries are 0 (never read: they lie beyond ``seq_lens``).
    """
    pages = (np.asarray(lens, np.int64) + page - 1) // page
    total = int(pages.sum())
    perm = _rng(w.cfg, 6, layer).permutation(total).astype(np.int32)
    mp = int(pages.max())
    bt = np.zeros((len(lens), mp), np.int32)
    off = 0
    for b, n in enumerate(pages):
        bt[b, :n] = perm[off:off + n]
        off += n
    return bt, total


def slots_of(block_table_row: np.ndarray, positions: np.ndarray, page: int = PAGE) -> np.ndarray:
    """Slot ``page_id * page + offset`` of each token position of one sequence."""
    positions = np.asarray(positions, np.int64)
    return block_table_row[positions // page].astype(np.int64) * page + positions % page


def device_sequence_tokens(w: Workload, layer: int, b: int, L: int, device: str = "cuda"):
    """Tokens ``[0, L)`` of sequence ``b`` drawn on the GPU (for contexts too long
    to draw on the host): the same distributions as :func:`sequence_tokens`
    (content ``N(0, 1)`` with the outlier channels scaled; RoPE pairs
    ``N(0, sigma_i^2)`` rotated by the position angle), from a torch generator
    seeded by ``(cfg, layer, b)``; a different stream from the host recipe.
    Returns bf16 tensors ``c_kv [L, 512]``, ``k_rope [L, 64]`` on ``device``.
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed((1000 * w.cfg + 7) * 1_000_003 + layer * 65_537 + b)
    c = torch.randn((L, D_C), generator=gen, device=device, dtype=torch.float32)
    c[:, torch.from_numpy(outlier_channels(w)).to(device)] *= w.outlier_mult
    c_kv = c.to(torch.bfloat16)
    del c
    i = torch.arange(D_R // 2, device=device, dtype=torch.float64)
    sigma = (0.1 * 50.0 ** (i / 31.0)).to(torch.float32)
    xy = torch.randn((L, D_R // 2, 2), generator=gen, device=device, dtype=torch.float32) * sigma[None, :, None]
    theta = 10000.0 ** (-2.0 * i / D_R)
    ang = (torch.arange(L, device=device, dtype=torch.float64)[:, None] * theta[None, :]).to(torch.float32)
    cs, sn = torch.cos(ang), torch.sin(ang)
    kr = torch.empty((L, D_R), device=device, dtype=torch.float32)
    kr[:, 0::2] = xy[..., 0] * cs - xy[..., 1] * sn
    kr[:, 1::2] = xy[..., 0] * sn + xy[..., 1] * cs
    return c_kv, kr.to(torch.bfloat16)


def generate_sequences(w: Workload, layer: int, lens, batch=None, threads: int = 8):
    """Generate token data of many sequences in parallel; yields ``(b, c_kv, k_rope)``."""
    bs = list(range(w.B)) if batch is None else list(batch)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        futs = [(b, ex.submit(sequence_tokens, w, layer, b, int(lens[b]))) for b in bs]
        for b, f in futs:
            c, k = f.result()
            yield b, c, k

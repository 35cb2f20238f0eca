"""Structured decode inputs in which every key is individually visible.

Input generation only: bf16 bit patterns of tokens and queries, and the key
positions worth probing.  No attention or quantization arithmetic.

Tokens (``marker_tokens``): token t of a sequence carries a marker of value
V_t = 1 + ((37 t) mod 16) / 8 in content channel t mod 512, on a background of
seeded uniform noise in [-0.05, 0.05]; the RoPE key is seeded N(0, 0.25).  So
the content latent of every key is distinct, and so is its contribution to
the output.

Queries, two modes:
  * ``uniform``: q_lat = q_rope = 0.  Every logit is exactly 0, so every
    visible key weighs 1/n: out = (1/n) sum_t c_hat_t and lse = ln n, with n
    the visible-key count (Sec. 2.1, eq. mla_compact; the identical-logit case
    of the softmax).  A key dropped or counted twice moves lse by about 1/n
    and the output channel of its marker by about V_t / n.
  * ``needle``: row r of a sequence probes one key position p_r: q_lat of the
    row is NEEDLE_Q in channel p_r mod 512 and 0 elsewhere, q_rope = 0.  The
    probed key's logit is tau * NEEDLE_Q * V (about 42 V), the background's
    at most about 2, so the row's output is the probed key's latent (when it
    is visible), and a score taken from the wrong key, or a probed key that
    is lost, changes the whole output row.

``edge_positions`` lists the tile (16- and 32-key), page (64-key), split,
causal and protection edges of a sequence, which both the GPU tests and the
CPU mutation check use.
"""
from __future__ import annotations

import numpy as np

from paper_2609_36760_amd import synthetic as syn

NEEDLE_Q = 576.0          # exact in bf16
TILE = 32
PAGE = 64


def marker_tokens(L: int, seed: int):
    """``(c_kv [L, 512], k_rope [L, 64])`` bf16 bit patterns (module docstring)."""
    rng = np.random.default_rng(seed)
    c = rng.uniform(-0.05, 0.05, size=(L, 512)).astype(np.float32)
    t = np.arange(L)
    c[t, t % 512] = 1.0 + ((37 * t) % 16) / 8.0
    k = (0.5 * rng.standard_normal((L, 64))).astype(np.float32)
    return syn.f32_to_bf16_bits(c), syn.f32_to_bf16_bits(k)


def edge_positions(L: int, split_tokens: int = 0, s_q: int = 1, protect=None) -> np.ndarray:
    """Key positions at every tile (16- and 32-key), page and split edge of a
    sequence of length L (the first and last key of each range and their
    neighbours), and the s_q newest keys (the causal edge).  Under a BF16
    protection policy ``(sink, recent)`` also the edges of the protected set
    and of the key list a protected decode walks -- the packed tiles from the
    one holding token ``sink`` up to token L - recent - 1, then the protected
    positions in order -- cut into 32-key tiles and splits of that list."""
    pos = {0, 1, L - 1, L - 2, L - 3}
    steps = [16, TILE, PAGE] + ([split_tokens] if split_tokens else [])
    for step in steps:
        for e in range(step, L + step, step):
            pos.update((e - 1, e, e + 1))
    pos.update(range(L - s_q - 1, L))
    if protect is not None:
        sink, recent = protect
        pos.update((sink - 1, sink, sink + 1, L - recent - 1, L - recent, L - recent + 1))
        prot = sorted(set(range(min(sink, L))) | set(range(max(0, L - recent), L)))
        has_packed = L - recent > sink
        pk0 = sink // TILE if has_packed else 0
        n_pk = (L - recent + TILE - 1) // TILE - pk0 if has_packed else 0
        n_list = n_pk + (len(prot) + TILE - 1) // TILE
        cuts = set(range(0, n_list + 1))                  # list-tile boundaries
        for u in cuts:
            for d in (-1, 0, 1):
                if u < n_pk:
                    t = TILE * (pk0 + u) + d
                else:
                    j = TILE * (u - n_pk) + d
                    t = prot[j] if 0 <= j < len(prot) else -1
                pos.add(t)
    return np.asarray(sorted(p for p in pos if 0 <= p < L), np.int64)


def queries(mode: str, s_q: int, H: int, probes=None):
    """``(q_lat [s_q, H, 512], q_rope [s_q, H, 64])`` bf16 bits of one sequence.

    ``needle``: ``probes [s_q * H]`` is the probed key position of each row
    (row r = i * H + h)."""
    ql = np.zeros((s_q * H, 512), np.float32)
    qr = np.zeros((s_q * H, 64), np.float32)
    if mode == "needle":
        ql[np.arange(s_q * H), np.asarray(probes) % 512] = NEEDLE_Q
    elif mode != "uniform":
        raise ValueError(mode)
    return (syn.f32_to_bf16_bits(ql).reshape(s_q, H, 512), syn.f32_to_bf16_bits(qr).reshape(s_q, H, 64))


def probe_positions(L: int, s_q: int, H: int, split_tokens: int, seed: int, part: int = 0,
                    protect=None) -> np.ndarray:
    """The probed position of every row: the sequence's edge positions first
    -- chunk ``part`` of H of them; each query token's rows take the chunk
    rotated by i, so the newest keys are probed by every query token, visible
    to some and masked for others -- the remaining rows seeded random
    positions."""
    edges = edge_positions(L, split_tokens, s_q, protect)[part * H:(part + 1) * H]
    rng = np.random.default_rng(seed)
    out = np.empty(s_q * H, np.int64)
    for i in range(s_q):
        row = np.concatenate([edges, rng.integers(0, L, size=max(H - len(edges), 0))])[:H]
        out[i * H:(i + 1) * H] = np.roll(row, i)
    return out


def needle_parts(L: int, s_q: int, H: int, split_tokens: int, protect=None) -> int:
    """Copies of a sequence the needle mode needs so that every edge position
    is probed (H rows per query token probe H positions per copy)."""
    return -(-len(edge_positions(L, split_tokens, s_q, protect)) // H)


def make_inputs(mode: str, lens, s_q: int, H: int, split_tokens: int, seed: int, protect=None,
                with_probes: bool = False):
    """Explicit inputs ``(tokens, q_lat [B, ...], q_rope [B, ...])`` of a batch
    (the form ``DecodeRun(inputs=...)`` takes).  In needle mode a length
    appears in as many sequences as its edge positions need (each with the
    same tokens, probing the next H of them).  ``with_probes``: also return
    the edge positions each sequence's rows probe (all of them in uniform
    mode, where every row sees every key)."""
    tokens, qls, qrs, probed = [], [], [], []
    for j, L in enumerate(lens):
        L = int(L)
        parts = needle_parts(L, s_q, H, split_tokens, protect) if mode == "needle" else 1
        for part in range(parts):
            tokens.append(marker_tokens(L, seed * 1000 + j))
            probes = (probe_positions(L, s_q, H, split_tokens, seed * 1000 + 500 + j, part, protect)
                      if mode == "needle" else None)
            ql, qr = queries(mode, s_q, H, probes)
            qls.append(ql)
            qrs.append(qr)
            edges = edge_positions(L, split_tokens, s_q, protect)
            probed.append(edges if probes is None else np.intersect1d(edges, probes))
    if with_probes:
        return (tokens, np.stack(qls), np.stack(qrs)), probed
    return tokens, np.stack(qls), np.stack(qrs)


# The structured GPU cases: (name, kind, c_bits, meta, H, s_q, split_tokens,
# protect (sink, recent) or None, lens).  Lengths sit on and around tile, page
# and split edges; 16 and 32 heads run the narrow kernel.
CASES = [
    ("c4_h128_sq1_nosplit", "lowbit", 4, "fp16", 128, 1, 0, None, [1, 31, 32, 33, 64, 65, 97, 200, 517]),
    ("c4_h128_sq2_split64", "lowbit", 4, "fp16", 128, 2, 64, None, [2, 33, 64, 65, 66, 129, 300]),
    ("c4_h128_sq2_split96", "lowbit", 4, "fp16", 128, 2, 96, None, [2, 95, 96, 97, 98, 193, 640]),
    ("c2_h128_sq1_split32", "lowbit", 2, "fp16", 128, 1, 32, None, [5, 32, 33, 95, 290]),
    ("c4paper_h128_sq1_split64", "lowbit", 4, "paper", 128, 1, 64, None, [3, 63, 64, 65, 130, 400]),
    ("bf16_h128_sq2_split96", "bf16", 16, "fp16", 128, 2, 96, None, [2, 96, 97, 98, 260]),
    ("bf16_h128_sq1_nosplit", "bf16", 16, "fp16", 128, 1, 0, None, [1, 32, 33, 300]),
    ("prot4x128_c4_h128_sq1_split64", "lowbit", 4, "fp16", 128, 1, 64, (4, 128), [1, 4, 5, 132, 133, 161, 300]),
    ("prot40x8_c2_h128_sq2_split32", "lowbit", 2, "fp16", 128, 2, 32, (40, 8), [2, 40, 48, 49, 73, 333]),
    ("n_c4_h16_sq1_split32", "lowbit", 4, "fp16", 16, 1, 32, None, [1, 16, 17, 32, 33, 65, 200]),
    ("n_c2_h16_sq2_nosplit", "lowbit", 2, "fp16", 16, 2, 0, None, [2, 17, 33, 64, 65, 130]),
    ("n_c4_h32_sq1_split64", "lowbit", 4, "fp16", 32, 1, 64, None, [3, 63, 64, 65, 129]),
    ("n_bf16_h16_sq1_split32", "bf16", 16, "fp16", 16, 1, 32, None, [1, 31, 33, 96, 97]),
    ("n_prot4x128_c4_h16_sq1_split64", "lowbit", 4, "fp16", 16, 1, 64, (4, 128), [5, 132, 133, 200, 261]),
]

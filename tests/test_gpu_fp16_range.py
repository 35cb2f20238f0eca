"""The fp16 range of the low-bit datapath (GPU).

The low-bit decode kernels reconstruct the cache in fp16 and run fp16
products (the header's precondition: queries and dequantized latents within
the fp16 range).  Pinned here, on the 128-head and 16-head kernels, split and
unsplit, with all-zero queries (every visible key weighs the same, Sec. 2.1,
eq. mla_compact):

  * at the edge: latents whose dequantized values reach about 5.9e4 in
    magnitude match the oracle -- nothing between the fp16 tile and the bf16
    output overflows (fp32 products and sums, the fp16 split partials hold
    weighted means);
  * past it: a key one of whose dequantized latents exceeds the fp16 range
    (|x_hat| >= 65520) makes every row that sees it non-finite (its score is
    0 x inf, and its weight reaches every channel), output and lse alike --
    never a plausible finite value.  A row of the same work item that does
    not see it (the first query token, when the key is the newest) still
    multiplies the key's latents by its zero weight in the aggregation, so
    the key's overflowing channels come out non-finite there too; its other
    channels and its lse match the oracle, and so does every other sequence
    of the batch.
"""
import numpy as np
import pytest

from gpu_support import AttnStats, bf16_bits_to_f64, cache_values, compare_sequence, elem_bound, lse_bound
from oracle import attention as at
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

F16_OVERFLOW = 65520.0        # the smallest magnitude fp16 rounds to infinity


def _tokens(L, seed, big=None):
    """bf16 bits of L tokens: content uniform in [-5.5e4, 5.5e4]; ``big``
    (position, group): that token's content group holds +-1e5 instead."""
    rng = np.random.default_rng(seed)
    c = rng.uniform(-5.5e4, 5.5e4, size=(L, 512)).astype(np.float32)
    k = (0.5 * rng.standard_normal((L, 64))).astype(np.float32)
    if big is not None:
        t, grp = big
        c[t, 64 * grp:64 * grp + 64] = np.where(np.arange(64) % 2 == 0, 1e5, -1e5)
    return syn.f32_to_bf16_bits(c), syn.f32_to_bf16_bits(k)


CASES = [
    # (name, heads, split tokens)
    ("h128_nosplit", 128, 0),
    ("h128_split64", 128, 64),
    ("h16_nosplit", 16, 0),
    ("h16_split64", 16, 64),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fp16_range_edge_and_overflow(case):
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    name, H, split = case
    s_q = 2
    # sequence 0: values at the edge; 1: an overflowing key in the middle;
    # 2: the newest key overflows (seen by the second query token only)
    lens = [150, 150, 97]
    bigs = [None, (40, 3), (96, 5)]
    tokens = [_tokens(L, 900 + j, bigs[j]) for j, L in enumerate(lens)]
    ql = np.zeros((3, s_q, H, 512), np.uint16)
    qr = np.zeros((3, s_q, H, 64), np.uint16)
    w = syn.Workload(f"fp16_range_{name}", 900, B=3, H=H, s_q=s_q, context=None, layers=((4, 4),),
                     split_tokens=split, ctx_range=(1, 2))
    run = DecodeRun(w, kind="lowbit", inputs=(tokens, ql, qr))
    run.step()
    torch.cuda.synchronize()
    out = run.out.cpu().numpy()           # [B, s_q, H, 512] bf16 bits
    lse = run.lse.cpu().numpy()           # [B, s_q, H]
    stats = AttnStats()
    for b, L in enumerate(lens):
        c, k = cache_values(run, b)       # byte-exact cache check, then the stored values (fp64)
        over = np.abs(c) >= F16_OVERFLOW
        got = out[b].view(np.uint16).astype(np.uint32) << 16
        got = got.view(np.float32)
        if bigs[b] is None:
            assert not over.any() and np.abs(c).max() > 5.5e4, "edge values not reached"
            compare_sequence(stats, out[b], lse[b], ql[b], qr[b], c, k, run.tau, s_q)
            continue
        t, grp = bigs[b]
        assert over[t].any() and not np.delete(over, t, axis=0).any(), "overflow only in the planted key"
        # rows that see the key: query token i sees keys below L - s_q + i + 1
        for i in range(s_q):
            sees = t < L - s_q + i + 1
            if sees:
                assert not np.isfinite(got[i]).any(), f"{name} seq {b} token {i}: finite output past the fp16 range"
                assert not np.isfinite(lse[b, i]).any(), f"{name} seq {b} token {i}: finite lse past the fp16 range"
            else:
                # the key's overflowing channels are non-finite; the rest against
                # the oracle over the keys this row sees (the first t)
                bad = over[t]
                assert not np.isfinite(got[i][:, bad]).any(), f"{name} seq {b} token {i}: finite overflow channels"
                q1, r1 = ql[b, i:i + 1], qr[b, i:i + 1]
                want, want_lse = at.decode_sequence(q1, r1, c[:t], k[:t], run.tau)
                bound = lse_bound(q1, r1, c[:t], k[:t], run.tau, t, 1)
                tol = elem_bound(q1, r1, c[:t], k[:t], run.tau, t, 1, want, bound)
                g1 = bf16_bits_to_f64(out[b, i:i + 1])
                stats.add(g1[..., ~bad], want[..., ~bad], lse[b, i:i + 1], want_lse, bound, tol[..., ~bad])
    stats.check(f"fp16 range {name}")

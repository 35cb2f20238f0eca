"""The append-and-decode call against the two calls it replaces.

mla_lowbit_append_decode_attn (and the BF16 one) must leave exactly the cache
bytes of mla_lowbit_quant_append and return exactly the outputs of
mla_lowbit_decode_attn after it (+ the combine): the writer inside the decode
launch runs the same quantizer, and the decode reads the same bytes.  Cases
cover new tokens whose tile is staged in the prologue (short key ranges) and
later (long ranges), a split boundary between the two new tokens of a
sequence, two row blocks per work item (s_q = 2, 128 heads: both write the
same bytes), 4-bit, 2-bit and BF16 caches, the paper's metadata, and a
16-head shape (the writer then runs as its own launch).
"""
import numpy as np
import pytest

from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

CASES = [
    # (name, H, s_q, lens, kind, c_bits, meta, split_tokens)
    ("c4_sq1_split64", 128, 1, [1, 31, 33, 64, 200, 517], "lowbit", 4, "fp16", 64),
    ("c4_sq1_split512", 128, 1, [40, 513, 1500], "lowbit", 4, "fp16", 512),
    ("c4_sq2_split32_edge", 128, 2, [2, 33, 65, 300], "lowbit", 4, "fp16", 32),
    ("c4_sq2_nosplit", 128, 2, [2, 129, 250], "lowbit", 4, "fp16", 0),
    ("c2_sq1_split96", 128, 1, [5, 96, 97, 290], "lowbit", 2, "fp16", 96),
    ("c4_paper_sq1_split64", 128, 1, [3, 130, 400], "lowbit", 4, "paper", 64),
    ("c2_paper_sq2_nosplit", 128, 2, [2, 77, 191], "lowbit", 2, "paper", 0),
    ("bf16_sq1_split64", 128, 1, [1, 33, 300], "bf16", 16, "fp16", 64),
    ("bf16_sq2_nosplit", 128, 2, [2, 97, 260], "bf16", 16, "fp16", 0),
    ("c4_h16_narrow", 16, 1, [7, 256, 333], "lowbit", 4, "fp16", 64),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_append_decode_matches_separate_calls(case):
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    name, H, s_q, lens, kind, c_bits, meta, split = case
    w = syn.Workload(name, 150, B=len(lens), H=H, s_q=s_q, context=None,
                     layers=((c_bits if kind == "lowbit" else 4, 4),), split_tokens=split, ctx_range=(1, 2))
    lens = np.asarray(lens, np.int32)
    a = DecodeRun(w, kind=kind, seq_lens=lens, meta=meta)
    b = DecodeRun(w, kind=kind, seq_lens=lens, meta=meta)
    b.cache.copy_(a.cache)              # pages no token has reached hold whatever the allocation held
    torch.cuda.synchronize()
    a.step()
    b.fused_step()
    torch.cuda.synchronize()
    assert torch.equal(a.cache, b.cache), "cache bytes differ"
    assert torch.equal(a.out, b.out), "outputs differ"
    assert torch.equal(a.lse, b.lse), "lse differs"
    print(f"  {name}: cache {a.cache.numel()} bytes and {a.out.numel()} outputs identical", flush=True)

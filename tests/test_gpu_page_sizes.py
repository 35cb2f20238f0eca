"""GPU parity at cache page sizes other than 64 tokens.

The library takes any page size that is a multiple of 32 tokens (at most
2^20); the other GPU tests use the paper's 64.  Here the pages hold 32 tokens
(every 32-key tile is a page of its own, every 16-key tile of the 16-row
kernel half of one), 96 (not a power of two: tiles start at offsets 0, 32 and
64 of a page in turn, and key splits of 192 tokens end mid-page), 128 and 1024
tokens, through the writer, the decode launch and the step with the append
inside it, for the 128-row and 16-row kernels, INT4, INT2, the BF16 cache,
the paper's metadata record and BF16 protection of sink and recent tokens.
Each sequence's pages are read back and compared byte for byte with the
oracle's packing at the same page size (Appendix C.4; Appendix C.5, "Storage
layout"), and every output of every row with the oracle's attention over the
values those bytes hold (Sec. 2.1, eq. mla_compact), with the bounds of
``gpu_support``.
"""
import numpy as np
import pytest

from gpu_support import AttnStats, check_sequence, check_sequence_protected
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

CASES = [
    # (name, H, s_q, lens, cache, split_tokens, page_size, path, (sink, recent) or None)
    ("pg32_c4_h128_sq1_split64_fused", 128, 1, [1, 31, 32, 33, 95, 200], "c4", 64, 32, "fused", None),
    ("pg96_c4_h128_sq2_nosplit", 128, 2, [2, 95, 96, 97, 193, 300], "c4", 0, 96, "two-call", None),
    ("pg96_c2_h128_sq1_split192_fused", 128, 1, [5, 96, 191, 193, 400], "c2", 192, 96, "fused", None),
    ("pg128_bf16_h128_sq2_split64_fused", 128, 2, [2, 127, 129, 260], "bf16", 64, 128, "fused", None),
    ("pg32_c4_h16_sq1_split32_fused", 16, 1, [1, 17, 33, 130], "c4", 32, 32, "fused", None),
    ("pg96_c4_h16_sq2_nosplit", 16, 2, [2, 97, 290], "c4", 0, 96, "two-call", None),
    ("pg1024_c4_h16_sq1_split512_fused", 16, 1, [3, 1023, 1025, 2100], "c4", 512, 1024, "fused", None),
    ("pg1024_c4_h128_sq1_nosplit_fused", 128, 1, [1025, 1500], "c4", 0, 1024, "fused", None),
    ("pg32_c4paper_h128_sq1_split64", 128, 1, [1, 33, 200], "c4paper", 64, 32, "two-call", None),
    ("pg96_c4_h128_sq2_split32_prot_fused", 128, 2, [2, 133, 165, 300], "c4", 32, 96, "fused", (4, 128)),
    ("pg32_c4_h16_sq1_nosplit_prot_fused", 16, 1, [1, 131, 133, 400], "c4", 0, 32, "fused", (4, 128)),
]


def workload(case):
    name, H, s_q, lens, cache, split, page, path, prot = case
    bits = 2 if cache == "c2" else 4
    return syn.Workload(name, 500 + CASES.index(case), B=len(lens), H=H, s_q=s_q, context=None,
                        layers=((bits, 4),), split_tokens=split, ctx_range=(1, 2))


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_decode_page_size_all_rows(case):
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, H, s_q, lens, cache, split, page, path, prot = case
    policy = None if prot is None else mb.protect_policy(*prot)
    run = DecodeRun(workload(case), kind="bf16" if cache == "bf16" else "lowbit",
                    seq_lens=np.asarray(lens, np.int32), page_size=page, protect=policy,
                    meta="paper" if cache == "c4paper" else "fp16")
    assert run.page_bytes == (mb.mla_bf16_page_bytes(run.fmt) if cache == "bf16" else mb.mla_lowbit_page_bytes(run.fmt))
    if path == "fused":
        run.fused_step()
    else:
        run.step()
    torch.cuda.synchronize()
    stats = AttnStats()
    check = check_sequence if policy is None else check_sequence_protected
    for b in range(len(lens)):
        check(stats, run, b)
        print(f"  seq {b} L={lens[b]} page {page}: cumulative max_abs={stats.abs_max:.4g}", flush=True)
    stats.check(name)

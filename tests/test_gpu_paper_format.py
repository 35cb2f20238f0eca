"""GPU parity of decode over the paper's cache storage (bf16 content scales,
fp32 RoPE scales, byte zero-points; 320 B per token) against the oracle.

The writer's bytes are covered bit-exactly in ``test_gpu_writer.py``; here
every output of small ragged batches (4- and 2-bit content, one and two query
tokens, split and unsplit, with and without BF16 protection) and sampled
sequences of the 32 x 4096 benchmark shape are compared with the oracle's
exact attention over its own reconstruction from the same stored scales,
within the bounds of ``gpu_support``.
"""
import numpy as np
import pytest

from gpu_support import AttnStats, check_sequence, check_sequence_protected
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu


def _run(w, **kw):
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    run = DecodeRun(w, meta="paper", **kw)
    run.step()
    torch.cuda.synchronize()
    return run


SMALL = [
    # (name, H, s_q, c_bits, split_tokens, protect, lens)
    ("paper_c4_h128_sq1_nosplit", 128, 1, 4, 0, None, [1, 31, 32, 33, 200, 517]),
    ("paper_c4_h128_sq2_split64", 128, 2, 4, 64, None, [2, 65, 129, 300]),
    ("paper_c2_h128_sq1_split32", 128, 1, 2, 32, None, [5, 64, 290]),
    ("paper_c4_h16_sq2_nosplit", 16, 2, 4, 0, None, [2, 77, 257]),
    ("paper_c4_h128_sq2_prot_split96", 128, 2, 4, 96, (4, 128), [2, 132, 133, 165, 400]),
    ("paper_c2_h64_sq1_prot_nosplit", 64, 1, 2, 0, (4, 128), [1, 131, 140, 333]),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_paper_format_decode_small_all_rows(case):
    from paper_2609_36760_amd import _binding as mb
    name, H, s_q, cb, split, prot, lens = case
    w = syn.Workload(name, 400 + SMALL.index(case), B=len(lens), H=H, s_q=s_q, context=None,
                     layers=((cb, 4),), split_tokens=split, ctx_range=(1, 2))
    policy = None if prot is None else mb.protect_policy(*prot)
    run = _run(w, seq_lens=np.asarray(lens, np.int32), protect=policy)
    assert run.page_bytes == (20480 if cb == 4 else 12288)
    stats = AttnStats()
    for b in range(len(lens)):
        (check_sequence if prot is None else check_sequence_protected)(stats, run, b)
        print(f"  seq {b} L={lens[b]}: cumulative max_abs={stats.abs_max:.4g}", flush=True)
    stats.check(name)


@pytest.mark.slow
def test_paper_format_bench_shape_sampled():
    import torch
    w = syn.WORKLOADS["dsv3_b32_h128_4k_c4r4"]
    run = _run(w)
    stats = AttnStats()
    for b in (0, 16, 31):
        check_sequence(stats, run, b)
    stats.check("dsv3_b32_h128_4k_c4r4 paper storage")
    del run
    torch.cuda.empty_cache()

"""The allocation-free decode entry point against the decode + combine calls
it stands for (GPU).

mla_lowbit_decode_attn_noalloc keeps the split partials in the library's own
per-GPU storage and runs the combine itself; its outputs must equal, bit for
bit, those of mla_lowbit_decode_attn into caller-owned partials followed by
mla_splitkv_combine (the same kernels on the same inputs).  Two calls in a
row, the second smaller, show that nothing of the first call's partials leaks
into the second; unsplit and narrow (16-head) launches too.
"""
import numpy as np
import pytest

from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

CALLS = [
    # (name, H, s_q, lens, c_bits, split_tokens): consecutive calls, later ones smaller
    ("large", 128, 2, [4096, 3000, 2049, 513, 64, 2], 4, 256),
    ("smaller", 128, 1, [700, 33, 1], 4, 64),
    ("narrow", 16, 2, [300, 2], 2, 32),
    ("unsplit", 128, 1, [200, 31], 4, 0),
]


def _reference_and_noalloc(case):
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, H, s_q, lens, cb, split = case
    w = syn.Workload(f"noalloc_{name}", 500 + [c[0] for c in CALLS].index(name), B=len(lens), H=H, s_q=s_q,
                     context=None, layers=((cb, 4),), split_tokens=split, ctx_range=(1, 2))
    run = DecodeRun(w, seq_lens=np.asarray(lens, np.int32))
    run.step()                                     # writer, decode into run's partials, combine
    out = torch.full_like(run.out, 0x7F7F)
    lse = torch.full_like(run.lse, float("nan"))
    mb.mla_lowbit_decode_attn_noalloc(run.fmt, run.q_lat, run.q_rope, run.cache, run.num_pages, run.block_table,
                                      run.seq_lens, run.s_q, run.H, run.tau, split_tokens=run.split_tokens,
                                      split_indptr=run.split_indptr, num_splits=run.num_splits, out=out, lse=lse)
    torch.cuda.synchronize()
    return run, out, lse


def test_noalloc_matches_decode_and_combine_on_consecutive_calls():
    import torch
    for case in CALLS:
        run, out, lse = _reference_and_noalloc(case)
        assert torch.equal(out, run.out), f"{case[0]}: outputs differ"
        assert torch.equal(lse, run.lse), f"{case[0]}: lse differs"
        print(f"  {case[0]}: {run.num_splits} splits x {run.s_q * run.H} rows, {out.numel()} outputs identical",
              flush=True)

"""Decode steps captured in a HIP graph and replayed (GPU).

Serving loops and the latency protocol of ``bench.py`` replay the step from a
captured graph.  Every library call only launches kernels on the caller's
stream (no allocation, copy or memset), so a captured step must reproduce the
eager one exactly: here each step is run eagerly, its outputs (and the cache
and protection bytes it writes) kept, the outputs poisoned, the step captured,
and the graph replayed three times with unrelated eager work and a
synchronization between replays; after every replay the outputs, lse, cache
and protection buffers must equal the eager ones bit for bit.  The steps: the
append inside the decode launch, then the combine (128-row and 16-row kernels,
INT4 and BF16 caches, BF16 protection); the writer, decode and combine as
three calls; and the allocation-free entry point (its partials in the
library's static storage).
"""
import numpy as np
import pytest

from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

CASES = [
    # (name, H, s_q, lens, kind, split_tokens, (sink, recent) or None, path)
    ("wide_c4_split_fused", 128, 1, [33, 300, 1000], "lowbit", 256, None, "fused"),
    ("wide_c4_sq2_three_calls", 128, 2, [2, 129, 600], "lowbit", 128, None, "step"),
    ("wide_bf16_split_fused", 128, 1, [40, 700], "bf16", 256, None, "fused"),
    ("narrow_c2_split_fused", 16, 2, [17, 900], "c2", 128, None, "fused"),
    ("wide_c4_protected_fused", 128, 1, [5, 140, 800], "lowbit", 256, (4, 128), "fused"),
    ("narrow_c4_protected_fused", 16, 1, [3, 133, 500], "lowbit", 64, (4, 128), "fused"),
    ("wide_c4_noalloc", 128, 1, [100, 1200], "lowbit", 256, None, "noalloc"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_graph_replay_matches_eager(case):
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, H, s_q, lens, kind, split, prot, path = case
    bits = 2 if kind == "c2" else 4
    w = syn.Workload(name, 700 + CASES.index(case), B=len(lens), H=H, s_q=s_q, context=None,
                     layers=((bits, 4),), split_tokens=split, ctx_range=(1, 2))
    run = DecodeRun(w, kind="bf16" if kind == "bf16" else "lowbit", seq_lens=np.asarray(lens, np.int32),
                    protect=None if prot is None else mb.protect_policy(*prot))

    def step():
        if path == "fused":
            run.fused_step()
        elif path == "step":
            run.step()
        else:
            mb.mla_lowbit_decode_attn_noalloc(run.fmt, run.q_lat, run.q_rope, run.cache, run.num_pages,
                                              run.block_table, run.seq_lens, run.s_q, run.H, run.tau,
                                              split_tokens=run.split_tokens, split_indptr=run.split_indptr,
                                              num_splits=run.num_splits, out=run.out, lse=run.lse)

    def poison():
        run.out.fill_(0x7F7F)
        run.lse.fill_(float("nan"))

    step()
    torch.cuda.synchronize()
    want_out, want_lse, want_cache = run.out.clone(), run.lse.clone(), run.cache.clone()
    want_prot = run.prot.clone() if prot is not None else None
    poison()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        poison()
        scratch.mul_(1.0001).add_(rep)           # unrelated eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(run.out, want_out), f"{name}: outputs of replay {rep} differ"
        assert torch.equal(run.lse, want_lse), f"{name}: lse of replay {rep} differs"
        assert torch.equal(run.cache, want_cache), f"{name}: cache bytes after replay {rep} differ"
        if want_prot is not None:
            assert torch.equal(run.prot, want_prot), f"{name}: protection buffers after replay {rep} differ"
    print(f"  {name}: 3 replays identical to the eager step", flush=True)

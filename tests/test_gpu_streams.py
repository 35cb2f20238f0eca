"""Independent decode steps on two streams at once (GPU).

The library keeps no state between calls (beyond a per-thread copy of the
last HIP error and an armed timing-event pair, and the allocation-free entry
point's static storage, whose calls on one GPU must not overlap), so two steps
on different buffers may run concurrently on two streams.  Each step's outputs,
lse, cache and protection bytes after five interleaved launches on two streams
must equal those of the same steps run one after the other on one stream.
"""
import numpy as np
import pytest

from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu


def test_two_streams_match_sequential_steps():
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    wa = syn.Workload("streams_wide", 900, B=4, H=128, s_q=2, context=None, split_tokens=256, ctx_range=(1, 2))
    wb = syn.Workload("streams_narrow", 901, B=6, H=16, s_q=1, context=None, split_tokens=64, ctx_range=(1, 2))
    a = DecodeRun(wa, seq_lens=np.asarray([2, 300, 1500, 4000], np.int32))
    b = DecodeRun(wb, seq_lens=np.asarray([1, 70, 133, 900, 2500, 5000], np.int32), protect=mb.protect_policy())
    runs = (a, b)
    for r in runs:
        r.fused_step()
    torch.cuda.synchronize()
    want = [(r.out.clone(), r.lse.clone(), r.cache.clone()) for r in runs]
    want_prot = b.prot.clone()
    for r in runs:
        r.out.fill_(0x7F7F)
        r.lse.fill_(float("nan"))
    torch.cuda.synchronize()
    streams = (torch.cuda.Stream(), torch.cuda.Stream())     # default priority
    for _ in range(5):
        for r, s in zip(runs, streams):
            r.fused_step(stream=s)
    torch.cuda.synchronize()
    for r, (o, l, c), tag in zip(runs, want, ("wide", "narrow protected")):
        assert torch.equal(r.out, o), f"{tag}: outputs differ"
        assert torch.equal(r.lse, l), f"{tag}: lse differs"
        assert torch.equal(r.cache, c), f"{tag}: cache bytes differ"
    assert torch.equal(b.prot, want_prot), "protection buffers differ"
    print("  two streams: 5 interleaved steps each, identical to the sequential steps", flush=True)

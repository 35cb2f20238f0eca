"""GPU parity at a million tokens per sequence (sampled).

The paper's latency grid reaches 1M-token contexts; the full-size parity
tests stop at 128K.  Here 16 sequences of 2^20 tokens (a 5.2 GB packed cache,
pages a seeded permutation over all of it, so byte offsets well past 2^32)
run the step the benchmarks time (the new token written inside the decode
launch, then the combine): the 16-row kernel with the paper's sink/recent BF16
protection at 16 heads, and the 128-row kernel at 128 heads.  For the last
sequence the pages are read back and compared byte for byte with the oracle's
packing of the same tokens (drawn on the GPU by the seeded generator and
copied to the host), and the oracle's attention over those values is compared
with every output of the sampled heads, with the bounds of ``gpu_support``.
"""
import time

import numpy as np
import pytest

from gpu_support import AttnStats, check_sequence, check_sequence_protected
from paper_2609_36760_amd import synthetic as syn

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CASES = [
    # (name, H, split_tokens, (sink, recent) or None, sampled heads)
    ("h16_b16_1m_protected", 16, 16384, (4, 128), None),
    ("h128_b16_1m", 128, 65536, None, [0, 37, 64, 127]),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_million_token_sequences_sampled(case):
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, H, split, prot, heads = case
    t0 = time.perf_counter()
    w = syn.Workload(name, 800 + CASES.index(case), B=16, H=H, s_q=1, context=1 << 20, split_tokens=split)
    run = DecodeRun(w, device_tokens=True, protect=None if prot is None else mb.protect_policy(*prot))
    assert run.num_pages * run.page_bytes > 1 << 32
    run.fused_step()
    torch.cuda.synchronize()
    print(f"  {name}: {run.num_pages} pages ({run.num_pages * run.page_bytes / 1e9:.1f} GB), "
          f"{run.num_splits} splits, step done at {time.perf_counter() - t0:.0f} s", flush=True)
    stats = AttnStats()
    b = w.B - 1
    (check_sequence if prot is None else check_sequence_protected)(stats, run, b, heads)
    print(f"  {name}: sequence {b} checked at {time.perf_counter() - t0:.0f} s, "
          f"max_abs {stats.abs_max:.4g}", flush=True)
    stats.check(name)
    del run
    torch.cuda.empty_cache()

"""GPU parity on structured inputs in which every key is individually
visible (``structured.py``): with all-zero queries every visible key weighs
exactly 1/n, so the output is the mean of the visible latents and the lse is
ln n; with needle queries every row's output is the latent of the one key it
probes.  The marker latents make every key's contribution distinct, and the
lengths, splits and probed positions sit on every tile (16- and 32-key),
page, split, causal and protection edge.  A key dropped, counted twice, or
scored from its neighbour fails these cases
(``test_parity_sensitivity.py`` shows it on the CPU for every edge position).

Covered: the wide kernel (128 heads; INT4, INT2, the paper's metadata, BF16,
BF16 protection; one and two query tokens; split and unsplit) and the narrow
kernel (16 and 32 heads; INT4, INT2, BF16, protection).  The uniform mode
runs the separate writer launch, the needle mode (unprotected) the
append-and-decode call the benchmark times.
"""
import numpy as np
import pytest

import structured as st
from gpu_support import AttnStats, check_sequence, check_sequence_protected
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", ["uniform", "needle"])
@pytest.mark.parametrize("case", st.CASES, ids=[c[0] for c in st.CASES])
def test_structured_all_rows(case, mode):
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, kind, cb, meta, H, s_q, split, prot, lens = case
    seed = 700 + st.CASES.index(case)
    inputs = st.make_inputs(mode, lens, s_q, H, split, seed, prot)
    w = syn.Workload(f"{name}_{mode}", seed, B=len(inputs[0]), H=H, s_q=s_q, context=None,
                     layers=((cb if kind == "lowbit" else 4, 4),), split_tokens=split, ctx_range=(1, 2))
    policy = None if prot is None else mb.protect_policy(*prot)
    print(f"{name} {mode}: {w.B} sequences, lengths {[len(c) for c, _ in inputs[0]]}", flush=True)
    run = DecodeRun(w, kind=kind, meta=meta, protect=policy, inputs=inputs)
    if mode == "needle" and policy is None:
        run.fused_step()
    else:
        run.step()
    torch.cuda.synchronize()
    stats = AttnStats()
    for b in range(w.B):
        (check_sequence if policy is None else check_sequence_protected)(stats, run, b)
    stats.check(f"{name} {mode}")

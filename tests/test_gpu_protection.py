"""GPU parity of BF16 protection of sink and recent tokens against the oracle.

Writer: after a chunked prefill and a decode-step append through
``mla_lowbit_quant_append_protected``, every row of P_L in every protection
buffer holds the token's bf16 bits (the oracle's lifecycle, buffers reached
through a permuted slot map), and the packed pages are byte-identical to those
of the unprotected writer.

Decode: every output of ragged batches whose lengths sit on and around each
boundary of the policy -- every token protected, the sink/window overlap, the
first packed token, tile and split edges -- for one and two query tokens,
split and unsplit launches, 4- and 2-bit content and several policies, checked
against the oracle's single softmax over the per-token representations with
the bounds of ``gpu_support``; the benchmark shape with the paper's policy on
sampled sequences.
"""
import numpy as np
import pytest

from gpu_support import FP16_LIMITED, AttnStats, check_fp16_limited, check_sequence_protected
from oracle import protection as pr
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu


def _run(w, policy, **kw):
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    run = DecodeRun(w, protect=policy, **kw)
    run.step()
    torch.cuda.synchronize()
    return run


EDGE_LENS = [1, 3, 4, 5, 31, 32, 33, 100, 131, 132, 133, 134, 160, 161, 164, 165, 197, 517, 1000]


def test_writer_protection_rows_and_packed_pages():
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    lens = np.asarray(EDGE_LENS, np.int32)
    w = syn.Workload("prot_writer", 300, B=len(lens), H=16, s_q=2, context=None, ctx_range=(1, 2))
    lens = np.maximum(lens, 2)
    slots = np.random.default_rng(3).permutation(len(lens) + 3)[:len(lens)].astype(np.int32)
    pol = mb.protect_policy()
    run = DecodeRun(w, protect=pol, seq_lens=lens, prot_slots=slots, prefill=False)
    plain = DecodeRun(w, seq_lens=lens, prefill=False)
    for r in (run, plain):          # same fill, so untouched bytes compare equal too
        r.cache.fill_(0x5A)
        r._prefill(16)
        r.append_new_tokens()
    torch.cuda.synchronize()
    assert torch.equal(run.cache, plain.cache)
    prot = run.prot.cpu().numpy().view(np.uint16).reshape(run.num_prot, pol.sink + pol.recent, 576)
    for b, L in enumerate(lens):
        c, k = syn.sequence_tokens(w, 0, b, int(L))
        pos, cb, kb = pr.read_protection(prot[slots[b]], int(L), 512, pol.sink, pol.recent)
        np.testing.assert_array_equal(cb, c[pos])
        np.testing.assert_array_equal(kb, k[pos])
        # the same rows as the oracle's own lifecycle (prefill, then the step)
        buf = np.zeros((pol.sink + pol.recent, 576), np.uint16)
        hist = int(L) - 2
        pr.write_protection(buf, np.arange(hist), hist, c[:hist], k[:hist], pol.sink, pol.recent)
        pr.write_protection(buf, np.arange(hist, int(L)), int(L), c[hist:], k[hist:], pol.sink, pol.recent)
        rows = sorted({pr.buffer_row(int(p), pol.sink, pol.recent) for p in pos})
        np.testing.assert_array_equal(prot[slots[b]][rows], buf[rows])
    print(f"writer: {len(lens)} sequences, protection rows and packed pages match", flush=True)


SMALL = [
    # (name, H, s_q, c_bits, split_tokens, (sink, recent), lens)
    ("p4x128_c4_h128_sq1_nosplit", 128, 1, 4, 0, (4, 128), EDGE_LENS),
    ("p4x128_c4_h128_sq2_split32", 128, 2, 4, 32, (4, 128), [2, 5, 132, 133, 165, 300]),
    ("p4x128_c4_h128_sq1_split64", 128, 1, 4, 64, (4, 128), [1, 100, 133, 161, 260, 517]),
    ("p4x128_c4_h16_sq2_split96", 16, 2, 4, 96, (4, 128), [2, 131, 134, 197, 1000]),
    ("p4x128_c2_h128_sq2_nosplit", 128, 2, 2, 0, (4, 128), [2, 130, 133, 290]),
    ("p40x8_c4_h128_sq2_split32", 128, 2, 4, 32, (40, 8), [2, 40, 48, 49, 72, 73, 100, 333]),
    ("p0x64_c4_h64_sq1_nosplit", 64, 1, 4, 0, (0, 64), [1, 64, 65, 96, 97, 250]),
    ("p3x0_c4_h128_sq2_split64", 128, 2, 4, 64, (3, 0), [2, 3, 4, 5, 35, 200]),
    ("p1x1_c2_h48_sq2_nosplit", 48, 2, 2, 0, (1, 1), [2, 3, 33, 64, 65]),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_protected_decode_small_all_rows(case):
    from paper_2609_36760_amd import _binding as mb
    name, H, s_q, cb, split, (sink, recent), lens = case
    w = syn.Workload(name, 310 + SMALL.index(case), B=len(lens), H=H, s_q=s_q, context=None,
                     layers=((cb, 4),), split_tokens=split, ctx_range=(1, 2))
    run = _run(w, mb.protect_policy(sink, recent), seq_lens=np.asarray(lens, np.int32))
    stats = AttnStats()
    for b in range(len(lens)):
        check_sequence_protected(stats, run, b)
        print(f"  seq {b} L={lens[b]}: cumulative max_abs={stats.abs_max:.4g}", flush=True)
    stats.check(name)


@pytest.mark.slow
def test_protected_decode_bench_shape_sampled():
    """32 x 4096, 128 heads, split 512, the paper's policy: launch configuration
    of the benchmark's protected step."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    w = syn.WORKLOADS["dsv3_b32_h128_4k_c4r4"]
    run = _run(w, mb.protect_policy())
    stats = AttnStats()
    for b in (0, 13, 31):
        check_sequence_protected(stats, run, b)
    stats.check("dsv3_b32_h128_4k_c4r4 protected")
    del run
    torch.cuda.empty_cache()


def test_protected_decode_paper_attention_shape():
    """The paper's kernel configuration: 16 heads, one query token, C4R4 with
    sink 4 / recent 128, split key ranges; 8 sequences of 4096 tokens, every row."""
    from paper_2609_36760_amd import _binding as mb
    w = syn.Workload("paper_h16_b8_4k", 330, B=8, H=16, s_q=1, context=4096, split_tokens=256)
    run = _run(w, mb.protect_policy())
    stats = AttnStats()
    for b in range(w.B):
        check_sequence_protected(stats, run, b)
    stats.check("paper_h16_b8_4k protected")


def test_device_drawn_inputs_sixteen_heads():
    """Long-context inputs drawn on the GPU (the 16-head latency grid's path):
    prefill through the protected writer and decode, every row of two 3000-token
    sequences against the oracle on the same drawn tokens (copied to the host)."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    w = syn.Workload("dev_h16_b2_3000", 340, B=2, H=16, s_q=1, context=3000, split_tokens=256)
    run = DecodeRun(w, protect=mb.protect_policy(), device_tokens=True)
    run.step()
    torch.cuda.synchronize()
    stats = AttnStats()
    for b in range(w.B):
        check_sequence_protected(stats, run, b)
    stats.check("device-drawn 16 heads protected")


AGING = [
    # (name, c_bits, H, s_q, split_tokens, (sink, recent), start lengths, steps)
    ("aging_c4_h128_sq1_split64", 4, 128, 1, 64, (4, 128), [1, 4, 100, 127, 128, 129, 131, 200], 36),
    ("aging_c4_h128_sq2_nosplit", 4, 128, 2, 0, (4, 128), [2, 98, 126, 130, 164], 20),
    ("aging_c2_h128_sq2_split32", 2, 128, 2, 32, (40, 8), [2, 40, 47, 60], 16),
    ("aging_c4_h16_sq2_split32", 4, 16, 2, 32, (4, 128), [2, 100, 129, 133], 20),
]


@pytest.mark.parametrize("case", AGING, ids=[c[0] for c in AGING])
def test_token_aging_over_consecutive_steps(case):
    """Consecutive decode steps of sequences that grow across the recent
    window's edge (Appendix C.5, "BF16 protection and cache lifecycle"): each
    step appends s_q tokens through the protected writer (the token entering
    the window overwrites the ring row of the one leaving it, which attention
    then reads from its packed copy) and decodes.  After every step the whole
    protection buffer of every sequence equals the oracle's lifecycle replayed
    over the same calls, the packed pages equal the oracle's packing, and every
    output row matches the oracle's single softmax over the per-token
    representations."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, cb, H, s_q, split, (sink, recent), start, steps = case
    seed = 360 + AGING.index(case)
    cap = [L + s_q * (steps - 1) for L in start]
    w = syn.Workload(name, seed, B=len(start), H=H, s_q=s_q, context=None, layers=((cb, 4),),
                     split_tokens=split, ctx_range=(1, 2))
    tokens = [syn.sequence_tokens(w, 0, b, L) for b, L in enumerate(cap)]
    ql, qr = syn.queries(w, 0)
    run = DecodeRun(w, protect=mb.protect_policy(sink, recent), inputs=(tokens, ql, qr),
                    seq_lens=np.asarray(start, np.int32))
    rows = sink + recent
    bufs = []
    for b, L in enumerate(start):       # the oracle's lifecycle: the prefill call
        buf = np.zeros((rows, 576), np.uint16)
        hist = L - s_q
        pr.write_protection(buf, np.arange(hist), hist, tokens[b][0][:hist], tokens[b][1][:hist], sink, recent)
        bufs.append(buf)
    stats = AttnStats()
    for step in range(steps):
        if step:
            run.advance()
        run.step()
        torch.cuda.synchronize()
        prot = run.prot.cpu().numpy().view(np.uint16).reshape(run.num_prot, rows, 576)
        for b in range(w.B):
            L = int(run.lens[b])
            new = np.arange(L - s_q, L)
            pr.write_protection(bufs[b], new, L, tokens[b][0][new], tokens[b][1][new], sink, recent)
            assert np.array_equal(prot[run.prot_slot_host[b]], bufs[b]), \
                f"step {step}: protection buffer of sequence {b} (length {L}) differs from the oracle's ring"
            check_sequence_protected(stats, run, b)
        print(f"  step {step}: lengths {run.lens.tolist()}, buffers equal, "
              f"cumulative max_excess={stats.excess_max:.4g}", flush=True)
    if name in FP16_LIMITED:
        check_fp16_limited(stats, name)
    else:
        stats.check(name)

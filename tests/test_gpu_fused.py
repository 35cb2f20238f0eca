"""The append-and-decode call against the two calls it replaces.

mla_lowbit_append_decode_attn (and the BF16 one) must leave exactly the cache
bytes of mla_lowbit_quant_append and return exactly the outputs of
mla_lowbit_decode_attn after it (+ the combine): the writer inside the decode
launch runs the same quantizer, and the decode reads the same bytes.  Cases
cover new tokens whose tile is staged in the prologue (short key ranges) and
later (long ranges), a split boundary between the two new tokens of a
sequence, two row blocks per work item (s_q = 2, 128 heads: both write the
same bytes; four at 256 heads, and a part-filled second one at 80), 4-bit,
2-bit and BF16 caches, the paper's metadata, and the 16-row kernel (16 and 32
rows; s_q = 2 at 16 heads: two row blocks).
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
    ("c4_h16_sq2_split32_edge", 16, 2, [2, 17, 33, 65, 300], "lowbit", 4, "fp16", 32),
    ("c2_h16_sq1_nosplit", 16, 1, [5, 96, 290], "lowbit", 2, "fp16", 0),
    ("bf16_h16_sq2_split64", 16, 2, [2, 33, 300], "bf16", 16, "fp16", 64),
    ("c4_paper_h32_sq1_split32", 32, 1, [3, 130, 400], "lowbit", 4, "paper", 32),
    ("c4_h256_sq2_split64", 256, 2, [2, 65, 199], "lowbit", 4, "fp16", 64),
    ("c2_h80_sq2_nosplit", 80, 2, [2, 131, 260], "lowbit", 2, "fp16", 0),
    ("bf16_h256_sq2_split32", 256, 2, [2, 33, 100], "bf16", 16, "fp16", 32),
    ("c4_h32_sq1_split64", 32, 1, [1, 64, 65, 200], "lowbit", 4, "fp16", 64),
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


PROTECTED = [
    # (name, c_bits, meta, H, s_q, split_tokens, (sink, recent), start lengths, steps)
    ("prot_c4_h128_sq1_split64", 4, "fp16", 128, 1, 64, (4, 128), [1, 4, 100, 127, 128, 129, 131, 200], 6),
    ("prot_c4_h128_sq2_nosplit", 4, "fp16", 128, 2, 0, (4, 128), [2, 98, 126, 130, 164], 4),
    ("prot_c2_h128_sq2_split32", 2, "fp16", 128, 2, 32, (40, 8), [2, 40, 47, 60], 8),
    ("prot_c4_paper_h128_sq1_split32", 4, "paper", 128, 1, 32, (4, 16), [3, 20, 21, 90], 6),
    ("prot_c4_h128_sq2_recent1_split32", 4, "fp16", 128, 2, 32, (4, 1), [2, 6, 40, 70], 4),
    ("prot_c4_h128_sq1_sinkonly_split32", 4, "fp16", 128, 1, 32, (4, 0), [1, 3, 5, 70], 4),
    ("prot_c4_h16_sq2_split32", 4, "fp16", 16, 2, 32, (4, 128), [2, 100, 129, 133], 4),
    ("prot_c2_h16_sq1_split32", 2, "fp16", 16, 1, 32, (4, 16), [3, 20, 21, 90], 6),
    ("prot_c4_paper_h32_sq1_split64", 4, "paper", 32, 1, 64, (4, 128), [1, 100, 129, 200], 4),
    ("prot_c4_h16_sq2_recent1_split32", 4, "fp16", 16, 2, 32, (4, 1), [2, 6, 40, 70], 4),
    ("prot_c4_h256_sq2_split64", 4, "fp16", 256, 2, 64, (4, 128), [2, 126, 130, 200], 4),
]


@pytest.mark.parametrize("case", PROTECTED, ids=[c[0] for c in PROTECTED])
def test_protected_append_decode_matches_separate_calls(case):
    """mla_lowbit_append_decode_attn_protected against the protected writer
    followed by the protected decode, over consecutive steps across the
    window's edge: identical packed pages, protection buffers, outputs and
    lse after every step.  Cases: new tokens in a work item's first staged
    tiles and later, sequences still entirely protected, a protected phase
    that starts a work item, two row blocks (s_q = 2 at 128 heads), a one-row
    window (the older new token read packed), sink rows only, INT2, the
    paper's metadata, and the 16-row kernel (16 and 32 rows)."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    name, cb, meta, H, s_q, split, (sink, recent), start, steps = case
    cap = [L + s_q * (steps - 1) for L in start]
    w = syn.Workload(name, 170 + PROTECTED.index(case), B=len(start), H=H, s_q=s_q, context=None,
                     layers=((cb, 4),), split_tokens=split, ctx_range=(1, 2))
    tokens = [syn.sequence_tokens(w, 0, b, L) for b, L in enumerate(cap)]
    ql, qr = syn.queries(w, 0)
    lens = np.asarray(start, np.int32)
    pol = mb.protect_policy(sink, recent)
    a = DecodeRun(w, protect=pol, inputs=(tokens, ql, qr), seq_lens=lens, meta=meta)
    b = DecodeRun(w, protect=pol, inputs=(tokens, ql, qr), seq_lens=lens, meta=meta)
    b.cache.copy_(a.cache)
    b.prot.copy_(a.prot)
    torch.cuda.synchronize()
    for step in range(steps):
        if step:
            a.advance()
            b.advance()
        a.step()
        b.fused_step()
        torch.cuda.synchronize()
        assert torch.equal(a.cache, b.cache), f"step {step}: cache bytes differ"
        assert torch.equal(a.prot, b.prot), f"step {step}: protection buffers differ"
        assert torch.equal(a.out, b.out), f"step {step}: outputs differ"
        assert torch.equal(a.lse, b.lse), f"step {step}: lse differs"
    print(f"  {name}: {steps} steps, lengths {a.lens.tolist()}: cache, protection buffers and outputs identical",
          flush=True)


def test_timing_hook_leaves_outputs_and_times_the_kernel():
    """Events attached to the decode dispatch by mla_time_next_decode_launch:
    the outputs are unchanged, the pair is consumed by the decode dispatch (a
    second launch without re-arming records nothing new) and brackets a time
    shorter than events recorded around the call on the same stream."""
    import ctypes
    import os

    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    w = syn.Workload("hook", 150, B=4, H=128, s_q=1, context=None, layers=((4, 4),), split_tokens=256,
                     ctx_range=(1, 2))
    lens = np.asarray([300, 1000, 777, 1024], np.int32)
    a = DecodeRun(w, kind="lowbit", seq_lens=lens)
    b = DecodeRun(w, kind="lowbit", seq_lens=lens)
    b.cache.copy_(a.cache)
    torch.cuda.init()
    hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD | os.RTLD_GLOBAL)
    hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    ev = [ctypes.c_void_p() for _ in range(4)]
    for e in ev:
        assert hip.hipEventCreateWithFlags(ctypes.byref(e), 0) == 0

    def elapsed(x, y):
        f = ctypes.c_float()
        assert hip.hipEventElapsedTime(ctypes.byref(f), x, y) == 0
        return f.value

    try:
        sh = torch.cuda.current_stream().cuda_stream
        torch.cuda.synchronize()
        a.fused_step()
        mb.mla_time_next_decode_launch(ev[0].value, ev[1].value)
        assert hip.hipEventRecord(ev[2], sh) == 0
        b.fused_step()
        assert hip.hipEventRecord(ev[3], sh) == 0
        torch.cuda.synchronize()
        kern, window = elapsed(ev[0], ev[1]), elapsed(ev[2], ev[3])
        assert torch.equal(a.cache, b.cache) and torch.equal(a.out, b.out) and torch.equal(a.lse, b.lse)
        assert 0.0 < kern < window, (kern, window)
        # consumed: another launch leaves the pair as it was
        b.fused_step()
        torch.cuda.synchronize()
        assert elapsed(ev[0], ev[1]) == kern
        print(f"  kernel {kern * 1e3:.1f} us inside a {window * 1e3:.1f} us window", flush=True)
    finally:
        mb.mla_time_next_decode_launch(None, None)
        for e in ev:
            hip.hipEventDestroy(e)

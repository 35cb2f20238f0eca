"""Host-side checks of the C ABI (CPU only; no GPU work is launched).

The library must load, export every function include/mla_lowbit.h declares,
report the page geometry of the documented layout, plan splits as documented,
and reject invalid arguments on the host before any HIP call.
"""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mla_lowbit.h")


@pytest.fixture(scope="module")
def mb():
    from paper_2609_36760_amd import _binding
    if not os.path.exists(_binding.LIB_PATH):
        pytest.skip("libmla_lowbit.so not built (run __graft_entry__.build())")
    _binding.library()
    return _binding


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mla_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(mb):
    names = declared_functions()
    assert len(names) == 20
    lib = ctypes.CDLL(mb.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(mb.SYMBOLS) == names


def test_page_geometry(mb):
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=4)) == 20736
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=2)) == 12544
    assert mb.mla_bf16_page_bytes(mb.cache_format()) == 73728
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=4, page_size=32)) == 10496   # 10368 -> 256-aligned
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=3)) == -1
    assert mb.mla_lowbit_page_bytes(mb.cache_format(page_size=48)) == -1
    assert mb.mla_bf16_page_bytes(mb.cache_format(d_c=256)) == -1
    # the paper's metadata: 320 B per token, 20480 B per 64-token page
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=4, meta=mb.MLA_META_PAPER)) == 20480
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=2, meta=mb.MLA_META_PAPER)) == 12288
    assert mb.mla_lowbit_page_bytes(mb.cache_format(c_bits=4, page_size=32, meta=mb.MLA_META_PAPER)) == 10240
    assert mb.mla_lowbit_page_bytes(mb.cache_format(meta=2)) == -1
    assert mb.mla_bf16_page_bytes(mb.cache_format(meta=2)) == 73728      # the BF16 cache ignores it


def test_planner(mb):
    lens = np.array([1, 2048, 2049, 131072, 4095], np.int32)
    indptr, total = mb.mla_plan_splits(lens, 2048)
    assert indptr.tolist() == [0, 1, 2, 4, 68, 70]
    assert total == 70
    with pytest.raises(mb.MlaError):
        mb.mla_plan_splits(lens, 100)               # not a multiple of 32
    with pytest.raises(mb.MlaError):
        mb.mla_plan_splits(np.array([0], np.int32), 64)


def _decode_status(mb, **over):
    lib = mb.library()
    fmt = over.pop("fmt", mb.cache_format())
    args = dict(q_lat=16, q_rope=16, cache=256, num_pages=4, block_table=16, max_pages=2, seq_lens=16,
                B=1, s_q=1, H=128, scale=0.07, split_tokens=0, split_indptr=None, num_splits=0, out=16,
                lse=None, part_m=None, part_s=None, part_o=None)
    args.update(over)
    return lib.mla_lowbit_decode_attn(ctypes.byref(fmt), args["q_lat"], args["q_rope"], args["cache"],
                                      args["num_pages"], args["block_table"], args["max_pages"], args["seq_lens"],
                                      args["B"], args["s_q"], args["H"], args["scale"], args["split_tokens"],
                                      args["split_indptr"], args["num_splits"], args["out"], args["lse"],
                                      args["part_m"], args["part_s"], args["part_o"], None)


@pytest.mark.parametrize("over,status", [
    (dict(q_lat=None), 1), (dict(cache=None), 1), (dict(out=None), 1), (dict(s_q=3), 1), (dict(s_q=0), 1),
    (dict(H=24), 1), (dict(H=0), 1), (dict(B=-1), 1), (dict(max_pages=0), 1), (dict(num_pages=0), 1),
    (dict(cache=272), 1), (dict(q_lat=8), 2), (dict(scale=float("inf")), 1), (dict(scale=0.0), 1), (dict(scale=-0.1), 1),
    (dict(split_tokens=64, split_indptr=16, part_m=16, part_s=16, part_o=None), 1),
    (dict(split_tokens=48, split_indptr=16, part_m=16, part_s=16, part_o=16), 2),
    (dict(fmt="c3"), 1), (dict(fmt="r2"), 1), (dict(fmt="m2"), 1), (dict(fmt="g32"), 2), (dict(fmt="p48"), 2), (dict(fmt="p40"), 1), (dict(fmt="dc256"), 2),
    (dict(B=0), 0), (dict(B=0, q_lat=None, cache=None, out=None), 0), (dict(B=0, s_q=3), 1),
])
def test_decode_rejects_before_any_hip_call(mb, over, status):
    fmts = {"c3": mb.cache_format(c_bits=3), "r2": mb.cache_format(r_bits=2),
            "g32": mb.cache_format(group=32), "p48": mb.cache_format(page_size=48),
            "p40": mb.cache_format(page_size=40),
            "dc256": mb.cache_format(d_c=256), "m2": mb.cache_format(meta=2)}
    if "fmt" in over:
        over = dict(over, fmt=fmts[over["fmt"]])
    assert _decode_status(mb, **over) == status
    assert mb.mla_status_str(status).startswith("MLA_")


def test_append_and_combine_validation(mb):
    lib = mb.library()
    fmt = mb.cache_format()
    f = ctypes.byref(fmt)
    assert lib.mla_lowbit_quant_append(f, None, 512, 16, 64, 16, 4, 256, 1, None) == 1
    assert lib.mla_lowbit_quant_append(f, 16, 500, 16, 64, 16, 4, 256, 1, None) == 1     # stride < 512
    assert lib.mla_lowbit_quant_append(f, 16, 516, 16, 64, 16, 4, 256, 1, None) == 2     # stride % 8
    assert lib.mla_lowbit_quant_append(f, 18, 512, 16, 64, 16, 4, 256, 1, None) == 2     # misaligned rows
    assert lib.mla_lowbit_quant_append(f, 16, 512, 16, 64, 16, -1, 256, 1, None) == 1
    assert lib.mla_lowbit_quant_append(f, None, 512, None, 64, None, 0, None, 0, None) == 0   # n = 0
    assert lib.mla_bf16_append(f, 16, 512, 16, 64, 16, 4, 256, 0, None) == 1             # no pages
    assert lib.mla_splitkv_combine(16, 16, 16, 16, 1, 1, 3, 128, 512, 16, None, None) == 1
    assert lib.mla_splitkv_combine(16, 16, 16, 16, 1, 1, 1, 128, 256, 16, None, None) == 2
    assert lib.mla_splitkv_combine(16, 16, 16, 16, 0, 0, 1, 128, 512, 16, None, None) == 0
    assert lib.mla_splitkv_combine(16, 16, 16, 16, -1, 1, 1, 128, 512, 16, None, None) == 1   # negative split count
    assert lib.mla_last_hip_error() == 0


def test_protection_buffer_bytes(mb):
    fmt = mb.cache_format()
    assert mb.mla_protect_buffer_bytes(fmt, mb.protect_policy()) == 152064      # 132 rows x 1152 B
    assert mb.mla_protect_buffer_bytes(fmt, mb.protect_policy(0, 1)) == 1152
    assert mb.mla_protect_buffer_bytes(mb.cache_format(c_bits=2), mb.protect_policy(3, 0)) == 3456
    assert mb.mla_protect_buffer_bytes(fmt, mb.protect_policy(-1, 4)) == -1
    assert mb.mla_protect_buffer_bytes(fmt, mb.protect_policy(0, 0)) == -1
    assert mb.mla_protect_buffer_bytes(fmt, mb.protect_policy(0, 65537)) == -1
    assert mb.mla_protect_buffer_bytes(mb.cache_format(c_bits=3), mb.protect_policy()) == -1


def test_planner_protected(mb):
    """Tile lists (sink 4, recent 128): L=1 -> 1 protected tile; 132 -> 5 (every
    token protected); 133 -> 1 packed tile (tokens 4) + 5; 4096 -> 124 packed
    tiles (tokens 4..3967) + 5.  Policy (40, 8), L=100: packed tiles 1..2
    (tokens 40..91) + 2 tiles of 48 protected rows."""
    lens = np.array([1, 132, 133, 4096], np.int32)
    pol = mb.protect_policy()
    indptr, total = mb.mla_plan_splits_protected(lens, 32, pol)
    assert indptr.tolist() == [0, 1, 6, 12, 141] and total == 141
    indptr, total = mb.mla_plan_splits_protected(lens, 512, pol)
    assert indptr.tolist() == [0, 1, 2, 3, 12] and total == 12
    indptr, total = mb.mla_plan_splits_protected(np.array([100], np.int32), 32, mb.protect_policy(40, 8))
    assert total == 4
    with pytest.raises(mb.MlaError):
        mb.mla_plan_splits_protected(lens, 48, pol)
    with pytest.raises(mb.MlaError):
        mb.mla_plan_splits_protected(lens, 64, mb.protect_policy(-1, 2))
    with pytest.raises(mb.MlaError):
        mb.mla_plan_splits_protected(np.array([0], np.int32), 64, pol)


def _prot_decode_status(mb, pol, prot=256, prot_slot=16, num_prot=1):
    lib = mb.library()
    fmt = mb.cache_format()
    return lib.mla_lowbit_decode_attn_protected(ctypes.byref(fmt), ctypes.byref(pol), 16, 16, 256, 4, 16, 2, 16,
                                                1, 1, 128, 0.07, prot, num_prot, prot_slot, 0, None, 0, 16, None,
                                                None, None, None, None)


def test_protected_entry_points_reject_before_any_hip_call(mb):
    pol = mb.protect_policy()
    assert _prot_decode_status(mb, mb.protect_policy(-1, 4)) == 1
    assert _prot_decode_status(mb, mb.protect_policy(0, 0)) == 1
    assert _prot_decode_status(mb, pol, prot=None) == 1
    assert _prot_decode_status(mb, pol, prot_slot=None) == 1
    assert _prot_decode_status(mb, pol, num_prot=0) == 1
    assert _prot_decode_status(mb, pol, num_prot=-1) == 1
    assert _prot_decode_status(mb, pol, prot=264) == 2                   # not 16-byte aligned
    lib = mb.library()
    fmt = mb.cache_format()
    f, p = ctypes.byref(fmt), ctypes.byref(pol)
    good = dict(token_seq=16, positions=16, seq_lens=16, prot_slot=16, B=1, prot=256, num_prot=1)

    def app(**over):
        a = dict(good, **over)
        return lib.mla_lowbit_quant_append_protected(f, p, 16, 512, 16, 64, 16, 4, 256, 1, a["token_seq"],
                                                     a["positions"], a["seq_lens"], a["prot_slot"], a["B"],
                                                     a["prot"], a["num_prot"], None)
    assert app(token_seq=None) == 1
    assert app(prot=None) == 1
    assert app(B=0) == 1
    assert app(num_prot=0) == 1
    assert app(prot=260) == 2
    bad = mb.protect_policy(5, -1)
    assert lib.mla_lowbit_quant_append_protected(f, ctypes.byref(bad), 16, 512, 16, 64, 16, 4, 256, 1, 16, 16, 16,
                                                 16, 1, 256, 1, None) == 1
    # n = 0 is a no-op once the policy is valid
    assert lib.mla_lowbit_quant_append_protected(f, p, None, 512, None, 64, None, 0, None, 0, None, None, None,
                                                 None, 0, None, 0, None) == 0
    assert lib.mla_last_hip_error() == 0


def test_persistent_cache_bytes_reproduce_the_printed_ratios(mb):
    """eq. physical_cache_storage: 3.22x at 4K and 3.59x at 128K for the paper's
    storage (20480 + 8 B per page, 152064 B of protection) against BF16."""
    paper = mb.cache_format(c_bits=4, meta=mb.MLA_META_PAPER)
    bf16 = mb.cache_format(c_bits=16)
    pol = mb.protect_policy()
    assert mb.mla_persistent_cache_bytes(paper, pol, 64) == 20488 + 152064
    assert mb.mla_persistent_cache_bytes(paper, pol, 65) == 2 * 20488 + 152064
    assert mb.mla_persistent_cache_bytes(paper, None, 0) == 0
    for L, ratio in ((4096, 3.22), (131072, 3.59)):
        r = mb.mla_persistent_cache_bytes(bf16, None, L) / mb.mla_persistent_cache_bytes(paper, pol, L)
        assert round(r, 2) == ratio
    # the fp16-metadata layout: 20736 B pages
    assert mb.mla_persistent_cache_bytes(mb.cache_format(), None, 4096) == 64 * (20736 + 8)
    assert mb.mla_persistent_cache_bytes(paper, pol, -1) == -1
    assert mb.mla_persistent_cache_bytes(bf16, pol, 10) == -1
    assert mb.mla_persistent_cache_bytes(mb.cache_format(c_bits=3), None, 10) == -1


def _append_decode_status(mb, **over):
    lib = mb.library()
    fmt = mb.cache_format()
    args = dict(c_kv=16, c_stride=512, k_rope=16, k_stride=64, slots=16, q_lat=16, q_rope=16, cache=256,
                num_pages=4, block_table=16, max_pages=2, seq_lens=16, B=1, s_q=1, H=128, scale=0.07,
                split_tokens=0, split_indptr=None, num_splits=0, out=16, lse=None, part_m=None, part_s=None,
                part_o=None)
    args.update(over)
    return lib.mla_lowbit_append_decode_attn(
        ctypes.byref(fmt), args["c_kv"], args["c_stride"], args["k_rope"], args["k_stride"], args["slots"],
        args["q_lat"], args["q_rope"], args["cache"], args["num_pages"], args["block_table"], args["max_pages"],
        args["seq_lens"], args["B"], args["s_q"], args["H"], args["scale"], args["split_tokens"],
        args["split_indptr"], args["num_splits"], args["out"], args["lse"], args["part_m"], args["part_s"],
        args["part_o"], None)


@pytest.mark.parametrize("over,status", [
    (dict(c_kv=None), 1), (dict(slots=None), 1), (dict(c_stride=500), 1), (dict(c_kv=8), 2),
    (dict(k_stride=68), 2), (dict(q_lat=None), 1), (dict(out=8), 2), (dict(s_q=3), 1), (dict(H=24), 1),
    (dict(B=0), 0), (dict(B=0, c_kv=None, q_lat=None, cache=None, out=None), 0),
])
def test_append_decode_rejects_before_any_hip_call(mb, over, status):
    """The append-and-decode call validates the writer's and the decode's arguments on the host."""
    assert _append_decode_status(mb, **over) == status


def _prot_append_decode_status(mb, pol=None, fmt=None, **over):
    lib = mb.library()
    fmt = mb.cache_format() if fmt is None else fmt
    pol = mb.protect_policy() if pol is None else pol
    a = dict(c_kv=16, c_stride=512, k_rope=16, k_stride=64, slots=16, q_lat=16, q_rope=16, cache=256,
             num_pages=4, block_table=16, max_pages=2, seq_lens=16, B=1, s_q=1, H=128, scale=0.07, prot=256,
             num_prot=1, prot_slot=16, split_tokens=0, split_indptr=None, num_splits=0, out=16, lse=None,
             part_m=None, part_s=None, part_o=None)
    a.update(over)
    return lib.mla_lowbit_append_decode_attn_protected(
        ctypes.byref(fmt), ctypes.byref(pol), a["c_kv"], a["c_stride"], a["k_rope"], a["k_stride"], a["slots"],
        a["q_lat"], a["q_rope"], a["cache"], a["num_pages"], a["block_table"], a["max_pages"], a["seq_lens"],
        a["B"], a["s_q"], a["H"], a["scale"], a["prot"], a["num_prot"], a["prot_slot"], a["split_tokens"],
        a["split_indptr"], a["num_splits"], a["out"], a["lse"], a["part_m"], a["part_s"], a["part_o"], None)


@pytest.mark.parametrize("over,status", [
    (dict(c_kv=None), 1), (dict(slots=None), 1), (dict(c_stride=500), 1), (dict(c_kv=8), 2),
    (dict(q_lat=None), 1), (dict(out=8), 2), (dict(s_q=3), 1), (dict(H=24), 1),
    (dict(prot=None), 1), (dict(prot_slot=None), 1), (dict(num_prot=0), 1), (dict(prot=264), 2),
    (dict(B=0), 0),
])
def test_protected_append_decode_rejects_before_any_hip_call(mb, over, status):
    """The protected append-and-decode call validates the writer's, the
    protection's and the decode's arguments on the host."""
    assert _prot_append_decode_status(mb, **over) == status


def test_protected_append_decode_rejects_bad_policy_and_format(mb):
    assert _prot_append_decode_status(mb, pol=mb.protect_policy(-1, 4)) == 1
    assert _prot_append_decode_status(mb, pol=mb.protect_policy(0, 0)) == 1
    assert _prot_append_decode_status(mb, fmt=mb.cache_format(c_bits=16)) != 0
    assert mb.library().mla_last_hip_error() == 0


def test_timing_hook_takes_both_events_or_none(mb):
    """mla_time_next_decode_launch: a pair of events or two nulls (clear)."""
    lib = mb.library()
    assert lib.mla_time_next_decode_launch(16, None) == 1
    assert lib.mla_time_next_decode_launch(None, 16) == 1
    assert lib.mla_time_next_decode_launch(None, None) == 0


def test_noalloc_rejects_more_partials_than_its_storage(mb):
    """num_splits * s_q * H above 65536 partial rows: MLA_ENOTSUP before any
    HIP call (the pointers are never dereferenced)."""
    lib = mb.library()
    fmt = mb.cache_format()
    fake = 1 << 20                       # 256-byte aligned, never touched
    st = lib.mla_lowbit_decode_attn_noalloc(ctypes.byref(fmt), fake, fake, fake, 4, fake, 4, fake, 8, 2, 128, 0.1,
                                            64, fake, 257, fake, fake, None)
    assert st == mb.MLA_ENOTSUP
    st = lib.mla_lowbit_decode_attn_noalloc(ctypes.byref(fmt), fake, fake, fake, 4, fake, 4, fake, 8, 1, 128, 0.1,
                                            64, fake, 513, fake, fake, None)
    assert st == mb.MLA_ENOTSUP
    # scalar checks still apply
    st = lib.mla_lowbit_decode_attn_noalloc(ctypes.byref(fmt), fake, fake, fake, 4, fake, 4, fake, 8, 3, 128, 0.1,
                                            64, fake, 4, fake, fake, None)
    assert st == mb.MLA_EINVAL


# Launch sizes past a dispatch's 32-bit work-item count are refused on the
# host (only the refusing side is exercised: an accepted call would launch).
_SPLIT = dict(split_tokens=64, split_indptr=16, part_m=16, part_s=16, part_o=16)


@pytest.mark.parametrize("over", [
    dict(_SPLIT, num_splits=2 ** 24 - 7),              # 2^24 workgroups x 256 threads = 2^32
    dict(_SPLIT, num_splits=2 ** 23 - 7, s_q=2),       # two 128-row blocks
    dict(_SPLIT, num_splits=2 ** 23, H=256),
    dict(B=2 ** 24),                                   # unsplit: one work item per sequence
    dict(_SPLIT, num_splits=2 ** 26 - 7, H=16),        # 16-row kernel: 64-thread workgroups
    dict(_SPLIT, num_splits=2 ** 25 - 7, H=32),        # two 16-row blocks
    dict(_SPLIT, num_splits=2 ** 31 - 1),
    dict(_SPLIT, num_splits=2 ** 20, H=2 ** 30),       # rows beyond 32 bits
])
def test_decode_refuses_launches_past_one_dispatch(mb, over):
    assert _decode_status(mb, **over) == 2


def test_append_and_combine_refuse_launches_past_one_dispatch(mb):
    lib = mb.library()
    fmt = mb.cache_format()
    f = ctypes.byref(fmt)
    for fn in (lib.mla_lowbit_quant_append, lib.mla_bf16_append):
        assert fn(f, 16, 512, 16, 64, 16, 2 ** 25 + 1, 256, 1, None) == 2
        assert fn(f, 16, 512, 16, 64, 16, 2 ** 31 - 1, 256, 1, None) == 2
    # rows = B * s_q * H: 2^24 - 7 rounds up to 2^24 workgroups of 256 threads
    assert lib.mla_splitkv_combine(16, 16, 16, 16, 2 ** 17, 2 ** 17, 1, 128, 512, 16, None, None) == 2
    assert lib.mla_splitkv_combine(16, 16, 16, 16, 2 ** 20, 2 ** 16, 2, 128, 512, 16, None, None) == 2
    # the new tokens of an append-and-decode call
    assert _append_decode_status(mb, B=2 ** 24 + 1, s_q=2) == 2
    assert _prot_append_decode_status(mb, B=2 ** 25 + 1) == 2
    assert lib.mla_last_hip_error() == 0

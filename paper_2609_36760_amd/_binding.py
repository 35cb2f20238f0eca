"""ctypes binding of ``libmla_lowbit.so`` (declared in include/mla_lowbit.h).

Argument marshalling only: every function forwards device pointers of torch
tensors, sizes and the current HIP stream to the C entry point of the same
name and raises :class:`MlaError` on a non-zero status.  All computation runs
in the library's HIP kernels; nothing here computes on the host except the
split planner, which is itself a C entry point.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmla_lowbit.so")

MLA_OK, MLA_EINVAL, MLA_ENOTSUP, MLA_EHIP = 0, 1, 2, 3

SYMBOLS = (
    "mla_lowbit_page_bytes", "mla_bf16_page_bytes", "mla_lowbit_quant_append", "mla_bf16_append",
    "mla_plan_splits", "mla_lowbit_decode_attn", "mla_bf16_decode_attn", "mla_splitkv_combine",
    "mla_status_str", "mla_last_hip_error", "mla_protect_buffer_bytes", "mla_lowbit_quant_append_protected",
    "mla_plan_splits_protected", "mla_lowbit_decode_attn_protected", "mla_persistent_cache_bytes",
    "mla_lowbit_append_decode_attn", "mla_bf16_append_decode_attn", "mla_time_next_decode_launch",
    "mla_lowbit_decode_attn_noalloc", "mla_lowbit_append_decode_attn_protected",
)


class MlaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = f"{fn} failed: {mla_status_str(status)}"
        if status == MLA_EHIP:
            msg += f" (hipError {mla_last_hip_error()})"
        super().__init__(msg)


MLA_META_FP16, MLA_META_PAPER = 0, 1


class mla_cache_format(ctypes.Structure):
    _fields_ = [("d_c", ctypes.c_int32), ("d_r", ctypes.c_int32), ("group", ctypes.c_int32),
                ("c_bits", ctypes.c_int32), ("r_bits", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("meta", ctypes.c_int32)]


class mla_protect_policy(ctypes.Structure):
    _fields_ = [("sink", ctypes.c_int32), ("recent", ctypes.c_int32)]


def protect_policy(sink: int = 4, recent: int = 128) -> mla_protect_policy:
    """The paper's policy by default: 4 sink tokens and a 128-token window."""
    return mla_protect_policy(sink, recent)


def cache_format(c_bits: int = 4, page_size: int = 64, d_c: int = 512, d_r: int = 64,
                 group: int = 64, r_bits: int = 4, meta: int = MLA_META_FP16) -> mla_cache_format:
    return mla_cache_format(d_c, d_r, group, c_bits, r_bits, page_size, meta)


_lib = None


def library() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_36760_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    FMT = ctypes.POINTER(mla_cache_format)
    POL = ctypes.POINTER(mla_protect_policy)
    sig = {
        "mla_lowbit_page_bytes": (I64, [FMT]),
        "mla_bf16_page_bytes": (I64, [FMT]),
        "mla_lowbit_quant_append": (ctypes.c_int, [FMT, P, I64, P, I64, P, I32, P, I64, P]),
        "mla_bf16_append": (ctypes.c_int, [FMT, P, I64, P, I64, P, I32, P, I64, P]),
        "mla_plan_splits": (I32, [P, I32, I32, P]),
        "mla_lowbit_decode_attn": (ctypes.c_int, [FMT, P, P, P, I64, P, I32, P, I32, I32, I32, F32,
                                                  I32, P, I32, P, P, P, P, P, P]),
        "mla_bf16_decode_attn": (ctypes.c_int, [FMT, P, P, P, I64, P, I32, P, I32, I32, I32, F32,
                                                I32, P, I32, P, P, P, P, P, P]),
        "mla_splitkv_combine": (ctypes.c_int, [P, P, P, P, I32, I32, I32, I32, I32, P, P, P]),
        "mla_lowbit_append_decode_attn": (ctypes.c_int, [FMT, P, I64, P, I64, P, P, P, P, I64, P, I32, P, I32, I32,
                                                         I32, F32, I32, P, I32, P, P, P, P, P, P]),
        "mla_bf16_append_decode_attn": (ctypes.c_int, [FMT, P, I64, P, I64, P, P, P, P, I64, P, I32, P, I32, I32,
                                                       I32, F32, I32, P, I32, P, P, P, P, P, P]),
        "mla_protect_buffer_bytes": (I64, [FMT, POL]),
        "mla_persistent_cache_bytes": (I64, [FMT, POL, I64]),
        "mla_lowbit_quant_append_protected": (ctypes.c_int, [FMT, POL, P, I64, P, I64, P, I32, P, I64,
                                                             P, P, P, P, I32, P, I64, P]),
        "mla_plan_splits_protected": (I32, [P, I32, I32, POL, P]),
        "mla_lowbit_decode_attn_protected": (ctypes.c_int, [FMT, POL, P, P, P, I64, P, I32, P, I32, I32, I32, F32,
                                                            P, I64, P, I32, P, I32, P, P, P, P, P, P]),
        "mla_lowbit_append_decode_attn_protected": (ctypes.c_int, [FMT, POL, P, I64, P, I64, P, P, P, P, I64, P, I32,
                                                                   P, I32, I32, I32, F32, P, I64, P, I32, P, I32,
                                                                   P, P, P, P, P, P]),
        "mla_lowbit_decode_attn_noalloc": (ctypes.c_int, [FMT, P, P, P, I64, P, I32, P, I32, I32, I32, F32,
                                                          I32, P, I32, P, P, P]),
        "mla_status_str": (ctypes.c_char_p, [ctypes.c_int]),
        "mla_last_hip_error": (ctypes.c_int, []),
        "mla_time_next_decode_launch": (ctypes.c_int, [P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def mla_status_str(status: int) -> str:
    return library().mla_status_str(status).decode()


def mla_last_hip_error() -> int:
    return library().mla_last_hip_error()


def mla_time_next_decode_launch(start, stop) -> None:
    """Attach two HIP events (raw handles, or None for both) to this thread's
    next decode-kernel dispatch."""
    _check("mla_time_next_decode_launch", library().mla_time_next_decode_launch(start, stop))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(fn: str, status: int):
    if status != MLA_OK:
        raise MlaError(fn, status)


def mla_lowbit_page_bytes(fmt: mla_cache_format) -> int:
    return library().mla_lowbit_page_bytes(ctypes.byref(fmt))


def mla_bf16_page_bytes(fmt: mla_cache_format) -> int:
    return library().mla_bf16_page_bytes(ctypes.byref(fmt))


def mla_lowbit_quant_append(fmt, c_kv, k_rope, slot_mapping, cache, num_pages, stream=None):
    n = c_kv.shape[0]
    _check("mla_lowbit_quant_append", library().mla_lowbit_quant_append(
        ctypes.byref(fmt), _ptr(c_kv), c_kv.stride(0), _ptr(k_rope), k_rope.stride(0),
        _ptr(slot_mapping), n, _ptr(cache), num_pages, _stream(stream)))


def mla_bf16_append(fmt, c_kv, k_rope, slot_mapping, cache, num_pages, stream=None):
    n = c_kv.shape[0]
    _check("mla_bf16_append", library().mla_bf16_append(
        ctypes.byref(fmt), _ptr(c_kv), c_kv.stride(0), _ptr(k_rope), k_rope.stride(0),
        _ptr(slot_mapping), n, _ptr(cache), num_pages, _stream(stream)))


def mla_plan_splits(seq_lens, split_tokens: int):
    """Host planner; returns ``(split_indptr int32 [B+1], total_splits)``."""
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    indptr = np.zeros(lens.size + 1, dtype=np.int32)
    total = library().mla_plan_splits(lens.ctypes.data, lens.size, split_tokens, indptr.ctypes.data)
    if total < 0:
        raise MlaError("mla_plan_splits", -total)
    return indptr, int(total)


def _decode(name, fmt, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H, softmax_scale,
            split_tokens, split_indptr, num_splits, out, lse, part_m, part_s, part_o, stream):
    B = q_lat.shape[0]
    fn = getattr(library(), name)
    _check(name, fn(ctypes.byref(fmt), _ptr(q_lat), _ptr(q_rope), _ptr(cache), num_pages,
                    _ptr(block_table), block_table.shape[1], _ptr(seq_lens), B, s_q, H,
                    float(softmax_scale), split_tokens, _ptr(split_indptr), num_splits,
                    _ptr(out), _ptr(lse), _ptr(part_m), _ptr(part_s), _ptr(part_o), _stream(stream)))


def mla_lowbit_decode_attn(fmt, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H,
                           softmax_scale, split_tokens=0, split_indptr=None, num_splits=0, out=None,
                           lse=None, part_m=None, part_s=None, part_o=None, stream=None):
    _decode("mla_lowbit_decode_attn", fmt, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H,
            softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s, part_o, stream)


def mla_bf16_decode_attn(fmt, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H,
                         softmax_scale, split_tokens=0, split_indptr=None, num_splits=0, out=None,
                         lse=None, part_m=None, part_s=None, part_o=None, stream=None):
    _decode("mla_bf16_decode_attn", fmt, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H,
            softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s, part_o, stream)


def mla_lowbit_decode_attn_noalloc(fmt, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H,
                                   softmax_scale, split_tokens=0, split_indptr=None, num_splits=0, out=None,
                                   lse=None, stream=None):
    """Decode (+ combine when split) with the partials in the library's own
    storage; writes ``out`` and ``lse``."""
    B = q_lat.shape[0]
    _check("mla_lowbit_decode_attn_noalloc", library().mla_lowbit_decode_attn_noalloc(
        ctypes.byref(fmt), _ptr(q_lat), _ptr(q_rope), _ptr(cache), num_pages, _ptr(block_table),
        block_table.shape[1], _ptr(seq_lens), B, s_q, H, float(softmax_scale), split_tokens, _ptr(split_indptr),
        num_splits, _ptr(out), _ptr(lse), _stream(stream)))


def _append_decode(name, fmt, c_kv, k_rope, slot_mapping, q_lat, q_rope, cache, num_pages, block_table, seq_lens,
                   s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s, part_o,
                   stream):
    B = q_lat.shape[0]
    fn = getattr(library(), name)
    _check(name, fn(ctypes.byref(fmt), _ptr(c_kv), c_kv.stride(0), _ptr(k_rope), k_rope.stride(0),
                    _ptr(slot_mapping), _ptr(q_lat), _ptr(q_rope), _ptr(cache), num_pages,
                    _ptr(block_table), block_table.shape[1], _ptr(seq_lens), B, s_q, H,
                    float(softmax_scale), split_tokens, _ptr(split_indptr), num_splits,
                    _ptr(out), _ptr(lse), _ptr(part_m), _ptr(part_s), _ptr(part_o), _stream(stream)))


def mla_lowbit_append_decode_attn(fmt, c_kv, k_rope, slot_mapping, q_lat, q_rope, cache, num_pages, block_table,
                                  seq_lens, s_q, H, softmax_scale, split_tokens=0, split_indptr=None,
                                  num_splits=0, out=None, lse=None, part_m=None, part_s=None, part_o=None,
                                  stream=None):
    """The step's new tokens (rows b * s_q + i of c_kv / k_rope) appended, then decode."""
    _append_decode("mla_lowbit_append_decode_attn", fmt, c_kv, k_rope, slot_mapping, q_lat, q_rope, cache,
                   num_pages, block_table, seq_lens, s_q, H, softmax_scale, split_tokens, split_indptr, num_splits,
                   out, lse, part_m, part_s, part_o, stream)


def mla_bf16_append_decode_attn(fmt, c_kv, k_rope, slot_mapping, q_lat, q_rope, cache, num_pages, block_table,
                                seq_lens, s_q, H, softmax_scale, split_tokens=0, split_indptr=None,
                                num_splits=0, out=None, lse=None, part_m=None, part_s=None, part_o=None,
                                stream=None):
    _append_decode("mla_bf16_append_decode_attn", fmt, c_kv, k_rope, slot_mapping, q_lat, q_rope, cache,
                   num_pages, block_table, seq_lens, s_q, H, softmax_scale, split_tokens, split_indptr, num_splits,
                   out, lse, part_m, part_s, part_o, stream)


def mla_splitkv_combine(part_m, part_s, part_o, split_indptr, num_splits, B, s_q, H, out, lse=None, stream=None):
    _check("mla_splitkv_combine", library().mla_splitkv_combine(
        _ptr(part_m), _ptr(part_s), _ptr(part_o), _ptr(split_indptr), num_splits, B, s_q, H, 512,
        _ptr(out), _ptr(lse), _stream(stream)))


def mla_protect_buffer_bytes(fmt: mla_cache_format, policy: mla_protect_policy) -> int:
    return library().mla_protect_buffer_bytes(ctypes.byref(fmt), ctypes.byref(policy))


def mla_lowbit_quant_append_protected(fmt, policy, c_kv, k_rope, slot_mapping, cache, num_pages, token_seq,
                                      positions, seq_lens, prot_slot, prot, num_prot, stream=None):
    n = c_kv.shape[0]
    _check("mla_lowbit_quant_append_protected", library().mla_lowbit_quant_append_protected(
        ctypes.byref(fmt), ctypes.byref(policy), _ptr(c_kv), c_kv.stride(0), _ptr(k_rope), k_rope.stride(0),
        _ptr(slot_mapping), n, _ptr(cache), num_pages, _ptr(token_seq), _ptr(positions), _ptr(seq_lens),
        _ptr(prot_slot), seq_lens.shape[0], _ptr(prot), num_prot, _stream(stream)))


def mla_plan_splits_protected(seq_lens, split_tokens: int, policy: mla_protect_policy):
    """Host planner under protection; returns ``(split_indptr int32 [B+1], total_splits)``."""
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    indptr = np.zeros(lens.size + 1, dtype=np.int32)
    total = library().mla_plan_splits_protected(lens.ctypes.data, lens.size, split_tokens, ctypes.byref(policy),
                                                indptr.ctypes.data)
    if total < 0:
        raise MlaError("mla_plan_splits_protected", -total)
    return indptr, int(total)


def mla_lowbit_decode_attn_protected(fmt, policy, q_lat, q_rope, cache, num_pages, block_table, seq_lens, s_q, H,
                                     softmax_scale, prot, num_prot, prot_slot, split_tokens=0, split_indptr=None,
                                     num_splits=0, out=None, lse=None, part_m=None, part_s=None, part_o=None,
                                     stream=None):
    B = q_lat.shape[0]
    _check("mla_lowbit_decode_attn_protected", library().mla_lowbit_decode_attn_protected(
        ctypes.byref(fmt), ctypes.byref(policy), _ptr(q_lat), _ptr(q_rope), _ptr(cache), num_pages,
        _ptr(block_table), block_table.shape[1], _ptr(seq_lens), B, s_q, H, float(softmax_scale),
        _ptr(prot), num_prot, _ptr(prot_slot), split_tokens, _ptr(split_indptr), num_splits,
        _ptr(out), _ptr(lse), _ptr(part_m), _ptr(part_s), _ptr(part_o), _stream(stream)))


def mla_lowbit_append_decode_attn_protected(fmt, policy, c_kv, k_rope, slot_mapping, q_lat, q_rope, cache,
                                            num_pages, block_table, seq_lens, s_q, H, softmax_scale, prot,
                                            num_prot, prot_slot, split_tokens=0, split_indptr=None, num_splits=0,
                                            out=None, lse=None, part_m=None, part_s=None, part_o=None, stream=None):
    """The step's new tokens appended under protection, then decode."""
    B = q_lat.shape[0]
    _check("mla_lowbit_append_decode_attn_protected", library().mla_lowbit_append_decode_attn_protected(
        ctypes.byref(fmt), ctypes.byref(policy), _ptr(c_kv), c_kv.stride(0), _ptr(k_rope), k_rope.stride(0),
        _ptr(slot_mapping), _ptr(q_lat), _ptr(q_rope), _ptr(cache), num_pages, _ptr(block_table),
        block_table.shape[1], _ptr(seq_lens), B, s_q, H, float(softmax_scale), _ptr(prot), num_prot,
        _ptr(prot_slot), split_tokens, _ptr(split_indptr), num_splits, _ptr(out), _ptr(lse), _ptr(part_m),
        _ptr(part_s), _ptr(part_o), _stream(stream)))


def mla_persistent_cache_bytes(fmt: mla_cache_format, policy, L: int) -> int:
    """eq. physical_cache_storage for one request of ``L`` tokens (``policy``
    None: no protection)."""
    return library().mla_persistent_cache_bytes(ctypes.byref(fmt), None if policy is None else ctypes.byref(policy),
                                                int(L))

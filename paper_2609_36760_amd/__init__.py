"""Low-bit MLA decode for AMD MI355X (gfx950).

The compute lives in ``libmla_lowbit.so`` (HIP kernels behind the C ABI of
include/mla_lowbit.h); ``_binding`` forwards to it with the same names.
``synthetic`` draws seeded inputs; ``runner`` sets up device buffers and
runs whole decode steps through the binding.  Importing this package does not
load the library; the first binding call does, and fails loudly if it is not
built.
"""
from __future__ import annotations

_BINDING_NAMES = (
    "MlaError", "cache_format", "library", "mla_lowbit_page_bytes", "mla_bf16_page_bytes",
    "mla_lowbit_quant_append", "mla_bf16_append", "mla_plan_splits", "mla_lowbit_decode_attn",
    "mla_bf16_decode_attn", "mla_splitkv_combine", "mla_status_str", "mla_last_hip_error", "SYMBOLS",
)


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import _binding
        return getattr(_binding, name)
    raise AttributeError(name)

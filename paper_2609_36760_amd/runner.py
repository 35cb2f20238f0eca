"""Device-side setup and decode steps for a synthetic workload.

``DecodeRun`` owns the device buffers of one cache layer: the paged cache
(packed low-bit or BF16), page table, sequence lengths, queries, the split
plan and the partial/output buffers.  Building it prefills every sequence's
history through the library's own writer; ``step()`` then runs one pass of
the decode hot path: append the step's new tokens with the writer, decode
attention over the cache, and (when split) the split-KV combine.  Only the
binding is called; no result is computed on the host.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import _binding as mb
from . import synthetic as syn


def _dev(a, device):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class DecodeRun:
    def __init__(self, w: syn.Workload, layer: int = 0, kind: str = "lowbit", device: str = "cuda",
                 split_tokens: int | None = None, seq_lens=None, threads: int = 16, prefill: bool = True,
                 token_cache: dict | None = None, protect=None, prot_slots=None, meta: str = "fp16",
                 device_tokens: bool = False, inputs=None, page_size: int = syn.PAGE):
        """``protect``: an ``mla_protect_policy`` to keep sink/recent tokens in
        bf16 (low-bit caches only); ``prot_slots``: the protection buffer of
        each sequence (default: buffer b for sequence b); ``meta``: "fp16"
        (fp16 scale and zero) or "paper" (the paper's bf16 / fp32 scales);
        ``device_tokens``: draw the tokens on the GPU
        (:func:`synthetic.device_sequence_tokens`, for long contexts);
        ``inputs``: explicit host inputs ``(tokens, q_lat, q_rope)`` instead of
        the workload's seeded draws -- ``tokens[b] = (c_kv [L_b, 512],
        k_rope [L_b, 64])`` bf16 bit patterns of every position of sequence b
        (the last s_q are the step's new tokens), ``q_lat [B, s_q, H, 512]``,
        ``q_rope [B, s_q, H, 64]`` bf16 bit patterns.  With explicit inputs,
        ``seq_lens`` may start the sequences at a prefix of their tokens:
        pages are allocated for all of them and :meth:`advance` moves the
        sequences on, step by step.  ``page_size``: tokens per cache page (a
        multiple of 32)."""
        if inputs is not None and device_tokens:
            raise ValueError("explicit inputs are host arrays")
        self.inputs = inputs
        if kind not in ("lowbit", "bf16"):
            raise ValueError(kind)
        if protect is not None and kind != "lowbit":
            raise ValueError("protection applies to low-bit caches")
        self.protect = protect
        self.w, self.layer, self.kind, self.device = w, layer, kind, device
        self.c_bits, self.r_bits = w.layers[layer]
        if meta not in ("fp16", "paper"):
            raise ValueError(meta)
        self.meta = meta
        self.page_size = page_size
        self.fmt = mb.cache_format(c_bits=self.c_bits, page_size=page_size,
                                   meta=mb.MLA_META_PAPER if meta == "paper" else mb.MLA_META_FP16)
        self.B, self.H, self.s_q = w.B, w.H, w.s_q
        self.tau = w.tau
        if inputs is not None:
            capacity = np.asarray([len(c) for c, _ in inputs[0]], np.int32)
            lens = capacity if seq_lens is None else np.asarray(seq_lens, np.int32)
            if np.any(lens > capacity) or np.any(lens < self.s_q):
                raise ValueError("seq_lens must lie between s_q and the explicit token counts")
        else:
            lens = syn.seq_lens(w) if seq_lens is None else np.asarray(seq_lens, np.int32)
            capacity = lens
        self.lens = lens
        self.capacity = capacity
        bt, num_pages = syn.page_table(w, capacity, layer, page=page_size)
        self.block_table_host = bt
        self.num_pages = num_pages
        self.page_bytes = (mb.mla_lowbit_page_bytes(self.fmt) if kind == "lowbit"
                           else mb.mla_bf16_page_bytes(self.fmt))
        self.cache = torch.empty(num_pages * self.page_bytes, dtype=torch.uint8, device=device)
        self.block_table = _dev(bt, device)
        self.seq_lens = _dev(lens, device)
        ql, qr = syn.queries(w, layer) if inputs is None else (np.asarray(inputs[1], np.uint16),
                                                                  np.asarray(inputs[2], np.uint16))
        self.q_lat = _dev(ql.view(np.int16), device)
        self.q_rope = _dev(qr.view(np.int16), device)
        if protect is not None:
            slots = np.arange(self.B, dtype=np.int32) if prot_slots is None else np.asarray(prot_slots, np.int32)
            self.num_prot = int(slots.max()) + 1
            self.prot_bytes = mb.mla_protect_buffer_bytes(self.fmt, protect)
            self.prot = torch.zeros(self.num_prot * self.prot_bytes, dtype=torch.uint8, device=device)
            self.prot_slot_host = slots
            self.prot_slot = _dev(slots, device)
        self.split_tokens = w.split_tokens if split_tokens is None else split_tokens
        self.part_m = self.part_s = self.part_o = None
        self._plan()
        self.out = torch.empty((self.B, self.s_q, self.H, 512), dtype=torch.int16, device=device)
        self.lse = torch.empty((self.B, self.s_q, self.H), dtype=torch.float32, device=device)
        self.device_tokens = device_tokens
        self._step_tokens()
        if protect is not None:
            self.new_seq = _dev(np.repeat(np.arange(self.B, dtype=np.int32), self.s_q), device)
            hist = np.maximum(lens.astype(np.int64) - self.s_q, 0).astype(np.int32)
            self.hist_lens = _dev(hist, device)
        self.token_cache = token_cache
        if device_tokens:
            self._device_fill(prefill)
        elif prefill:
            self._prefill(threads)

    def _plan(self):
        """Split plan and partial buffers for the current lengths."""
        lens, device = self.lens, self.device
        if not self.split_tokens:
            self.split_indptr = self.part_m = self.part_s = self.part_o = None
            self.num_splits = 0
            return
        if self.protect is not None:
            indptr, total = mb.mla_plan_splits_protected(lens, self.split_tokens, self.protect)
        else:
            indptr, total = mb.mla_plan_splits(lens, self.split_tokens)
        self.split_indptr_host = indptr
        self.split_indptr = _dev(indptr, device)
        self.num_splits = total
        R = self.s_q * self.H
        if self.part_m is None or self.part_m.numel() < total * R:
            self.part_m = torch.empty(total * R, dtype=torch.float32, device=device)
            self.part_s = torch.empty(total * R, dtype=torch.float32, device=device)
            self.part_o = torch.empty(total * R * 512, dtype=torch.float16, device=device)

    def _step_tokens(self):
        """Slots, positions and host rows of the step's new tokens (the last s_q
        positions of every sequence)."""
        lens, bt, device = self.lens, self.block_table_host, self.device
        new_slots = [syn.slots_of(bt[b], np.arange(int(lens[b]) - self.s_q, int(lens[b])), self.page_size) for b in range(self.B)]
        self.new_slots = _dev(np.concatenate(new_slots), device)
        if not self.device_tokens:
            new_c, new_k = [], []
            for b in range(self.B):
                c, k = self.tokens(b, start=int(lens[b]) - self.s_q)
                new_c.append(c)
                new_k.append(k)
            self.new_c = _dev(np.concatenate(new_c).view(np.int16), device)
            self.new_k = _dev(np.concatenate(new_k).view(np.int16), device)
        self.new_pos = _dev(np.concatenate([np.arange(int(l) - self.s_q, int(l), dtype=np.int32) for l in lens]),
                            device)

    def advance(self):
        """Move every sequence on by s_q positions (explicit inputs): the next
        decode step's lengths, new tokens, slots and split plan.  The cache and
        protection buffers keep what earlier steps wrote."""
        if self.inputs is None:
            raise ValueError("advance() needs explicit inputs")
        lens = self.lens + self.s_q
        if np.any(lens > self.capacity):
            raise ValueError("no explicit tokens left to advance into")
        self.lens = lens.astype(np.int32)
        self.seq_lens = _dev(self.lens, self.device)
        self._plan()
        self._step_tokens()

    def tokens(self, b: int, start: int = 0):
        """Host bf16 bit patterns of positions ``[start, L_b)`` of sequence b:
        ``(c_kv, k_rope)`` from the explicit inputs or the workload's draw."""
        L = int(self.lens[b])
        if self.inputs is not None:
            c, k = self.inputs[0][b]
            return np.asarray(c[start:L], np.uint16), np.asarray(k[start:L], np.uint16)
        if self.device_tokens:
            c, k = syn.device_sequence_tokens(self.w, self.layer, b, L, self.device)
            return (c[start:].view(torch.int16).cpu().numpy().view(np.uint16),
                    k[start:].view(torch.int16).cpu().numpy().view(np.uint16))
        return syn.sequence_tokens(self.w, self.layer, b, L, start=start)

    def queries(self, b: int):
        """Host bf16 bit patterns ``(q_lat [s_q, H, 512], q_rope [s_q, H, 64])``
        of sequence b."""
        if self.inputs is not None:
            return np.asarray(self.inputs[1][b], np.uint16), np.asarray(self.inputs[2][b], np.uint16)
        ql, qr = syn.queries(self.w, self.layer, batch=[b])
        return ql[0], qr[0]

    def _device_fill(self, prefill: bool):
        """Draw every sequence on the GPU, write its history, keep its last s_q tokens."""
        new_c, new_k = [], []
        for b in range(self.B):
            L = int(self.lens[b])
            hist = L - self.s_q
            c, k = syn.device_sequence_tokens(self.w, self.layer, b, L, self.device)
            new_c.append(c[hist:].clone())
            new_k.append(k[hist:].clone())
            if prefill and hist > 0:
                slots = _dev(syn.slots_of(self.block_table_host[b], np.arange(hist), self.page_size), self.device)
                seq = torch.full((hist,), b, dtype=torch.int32, device=self.device)
                pos = torch.arange(hist, dtype=torch.int32, device=self.device)
                self._append(c[:hist].view(torch.int16), k[:hist].view(torch.int16), slots, seq, pos)
            del c, k
        torch.cuda.synchronize()
        self.new_c = torch.cat(new_c).view(torch.int16)
        self.new_k = torch.cat(new_k).view(torch.int16)

    def _append(self, c, k, slots, seq=None, pos=None):
        if self.protect is not None:
            mb.mla_lowbit_quant_append_protected(self.fmt, self.protect, c, k, slots, self.cache, self.num_pages,
                                                 seq, pos, self.hist_lens, self.prot_slot, self.prot,
                                                 self.num_prot)
            return
        fn = mb.mla_lowbit_quant_append if self.kind == "lowbit" else mb.mla_bf16_append
        fn(self.fmt, c, k, slots, self.cache, self.num_pages)

    def _prefill(self, threads: int, chunk_tokens: int = 1 << 20):
        """Write every sequence's history (all but the step's s_q new tokens)."""
        pend_c, pend_k, pend_s, pend_b, pend_p, pend_n = [], [], [], [], [], 0

        def flush():
            nonlocal pend_c, pend_k, pend_s, pend_b, pend_p, pend_n
            if pend_n:
                self._append(_dev(np.concatenate(pend_c).view(np.int16), self.device),
                             _dev(np.concatenate(pend_k).view(np.int16), self.device),
                             _dev(np.concatenate(pend_s), self.device),
                             _dev(np.concatenate(pend_b), self.device), _dev(np.concatenate(pend_p), self.device))
                torch.cuda.synchronize()
            pend_c, pend_k, pend_s, pend_b, pend_p, pend_n = [], [], [], [], [], 0

        hist = np.maximum(self.lens.astype(np.int64) - self.s_q, 0)
        tc = self.token_cache
        key = (self.w.name, self.layer)
        if self.inputs is not None:
            source = ((b, c[:int(hist[b])], k[:int(hist[b])]) for b, (c, k) in enumerate(self.inputs[0]))
            tc = None
        elif tc is not None and key in tc:
            source = ((b, c, k) for b, (c, k) in enumerate(tc[key]))
        else:
            source = syn.generate_sequences(self.w, self.layer, hist, threads=threads)
            if tc is not None:
                tc[key] = []
        for b, c, k in source:
            if tc is not None and len(tc[key]) == b:
                tc[key].append((c, k))
            n = int(hist[b])
            if n == 0:
                continue
            pend_c.append(c)
            pend_k.append(k)
            pend_s.append(syn.slots_of(self.block_table_host[b], np.arange(n), self.page_size))
            pend_b.append(np.full(n, b, np.int32))
            pend_p.append(np.arange(n, dtype=np.int32))
            pend_n += n
            if pend_n >= chunk_tokens:
                flush()
        flush()

    def append_new_tokens(self, stream=None):
        if self.protect is not None:
            mb.mla_lowbit_quant_append_protected(self.fmt, self.protect, self.new_c, self.new_k, self.new_slots,
                                                 self.cache, self.num_pages, self.new_seq, self.new_pos,
                                                 self.seq_lens, self.prot_slot, self.prot, self.num_prot,
                                                 stream=stream)
            return
        fn = mb.mla_lowbit_quant_append if self.kind == "lowbit" else mb.mla_bf16_append
        fn(self.fmt, self.new_c, self.new_k, self.new_slots, self.cache, self.num_pages, stream=stream)

    def attend(self, stream=None):
        """Decode attention (+ combine when split); results in ``out``/``lse``."""
        if self.protect is not None:
            mb.mla_lowbit_decode_attn_protected(
                self.fmt, self.protect, self.q_lat, self.q_rope, self.cache, self.num_pages, self.block_table,
                self.seq_lens, self.s_q, self.H, self.tau, self.prot, self.num_prot, self.prot_slot,
                split_tokens=self.split_tokens, split_indptr=self.split_indptr, num_splits=self.num_splits,
                out=self.out, lse=self.lse, part_m=self.part_m, part_s=self.part_s, part_o=self.part_o,
                stream=stream)
        else:
            fn = mb.mla_lowbit_decode_attn if self.kind == "lowbit" else mb.mla_bf16_decode_attn
            fn(self.fmt, self.q_lat, self.q_rope, self.cache, self.num_pages, self.block_table, self.seq_lens,
               self.s_q, self.H, self.tau, split_tokens=self.split_tokens, split_indptr=self.split_indptr,
               num_splits=self.num_splits, out=self.out, lse=self.lse, part_m=self.part_m,
               part_s=self.part_s, part_o=self.part_o, stream=stream)
        if self.split_tokens:
            mb.mla_splitkv_combine(self.part_m, self.part_s, self.part_o, self.split_indptr, self.num_splits, self.B,
                                   self.s_q,
                                   self.H, self.out, self.lse, stream=stream)

    def step(self, stream=None):
        self.append_new_tokens(stream)
        self.attend(stream)

    def fused_step(self, stream=None):
        """The same step with the append inside the decode call."""
        if self.protect is not None:
            mb.mla_lowbit_append_decode_attn_protected(
                self.fmt, self.protect, self.new_c, self.new_k, self.new_slots, self.q_lat, self.q_rope, self.cache,
                self.num_pages, self.block_table, self.seq_lens, self.s_q, self.H, self.tau, self.prot,
                self.num_prot, self.prot_slot, split_tokens=self.split_tokens, split_indptr=self.split_indptr,
                num_splits=self.num_splits, out=self.out, lse=self.lse, part_m=self.part_m, part_s=self.part_s,
                part_o=self.part_o, stream=stream)
        else:
            fn = mb.mla_lowbit_append_decode_attn if self.kind == "lowbit" else mb.mla_bf16_append_decode_attn
            fn(self.fmt, self.new_c, self.new_k, self.new_slots, self.q_lat, self.q_rope, self.cache,
               self.num_pages, self.block_table, self.seq_lens, self.s_q, self.H, self.tau,
               split_tokens=self.split_tokens, split_indptr=self.split_indptr, num_splits=self.num_splits,
               out=self.out, lse=self.lse, part_m=self.part_m, part_s=self.part_s, part_o=self.part_o,
               stream=stream)
        if self.split_tokens:
            mb.mla_splitkv_combine(self.part_m, self.part_s, self.part_o, self.split_indptr, self.num_splits, self.B,
                                   self.s_q,
                                   self.H, self.out, self.lse, stream=stream)

    # ---- accounting -------------------------------------------------------
    def visible_pairs(self) -> int:
        """Number of valid (query row, key) pairs of one step."""
        L = self.lens.astype(np.int64)
        return int(self.H * sum(int(l) - self.s_q + 1 + i for l in L for i in range(self.s_q)))

    def flops(self) -> int:
        """Algorithmic flops of one step: 2 * (576 + 512) per valid (row, key) pair."""
        return 2 * (576 + 512) * self.visible_pairs()

    def cache_token_bytes(self) -> int:
        if self.kind == "bf16":
            return 1152
        return (512 * self.c_bits + 64 * self.r_bits) // 8 + (32 if self.meta == "paper" else 9 * 4)

    def key_bytes(self) -> int:
        """Bytes of every cached key once (under protection, the
        min(L, sink + recent) protected tokens as 1152-byte bf16 rows)."""
        L = self.lens.astype(np.int64)
        if self.protect is None:
            return int(L.sum()) * self.cache_token_bytes()
        n_prot = np.minimum(L, self.protect.sink + self.protect.recent)
        return int(((L - n_prot) * self.cache_token_bytes() + n_prot * 1152).sum())

    def cache_bytes_read(self) -> int:
        """Cache bytes attention reads per step (every key once per 128-row block)."""
        return self.key_bytes() * math.ceil(self.s_q * self.H / 128)

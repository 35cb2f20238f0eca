"""Benchmark of the low-bit MLA decode step on one MI355X.

A step is one pass of the decode hot path for one cache layer: the step's new
tokens quantized and appended inside the fused low-bit decode launch, decode
attention over the paged cache, and the split-KV combine.  The headline
workload is the 128-head INT4/INT4 decode batch of 64 sequences x 32768 tokens
(the target shape; 680 MB of packed cache per layer).  Successive steps
alternate between two resident layer caches, so no step finds the previous
one's bytes in the 256 MB last-level cache.

Printed: one JSON line (stdout) with whole-step decode tokens/s at that shape,
the decode kernel's roofline (live HIP-event timing of every timed launch on
its own dispatch: mean, median, p10, p90), the sustained clock and socket
power (the step run back to back for 1.5 s after the timed steps), the same
step over a BF16 cache (the unquantized comparison), the 32 x 4096 workload,
the paper's sink/recent BF16 protection at both shapes, the paper's sampling
protocol (graph replay, caches flushed before every sample, 2 runs x 2 rounds
x 30 samples in alternating order), and the CPU oracle timed on a bounded
sample of the headline workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode attn tokens/s + HBM GB/s & MFMA util vs peak, 128 heads, INT4/INT4 vs BF16"
MAIN = "c4r4_b64_h128_32k"            # the headline: 64 x 32768, INT4/INT4, 128 heads
SMALL = "dsv3_b32_h128_4k_c4r4"       # 32 x 4096
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
LAYERS = {MAIN: 2, SMALL: 8}       # resident layer caches cycled by the timed steps


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class TimingEvents:
    """A pair of HIP timing events per timed decode launch.  ``arm(i)`` hands
    pair i to ``mla_time_next_decode_launch``: the library attaches it to the
    decode kernel's own dispatch (hipExtLaunchKernel), on the launch's stream,
    so the pair brackets the kernel's execution and not the dispatch latency
    that events recorded around the call would add (about 6 us per launch at
    32 x 4K).  The events are created with ``hipEventDisableSystemFence``, the
    runtime's flag for events used only to measure time (no system-scope cache
    writeback when their timestamp is written).  The HIP runtime is the one
    torch loaded (same soname); the events are destroyed with the object."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n: int):
        import ctypes
        import torch
        torch.cuda.init()
        self._c = ctypes
        hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD | os.RTLD_GLOBAL)
        hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self._hip = hip
        self.pairs = []
        for _ in range(n):
            pair = []
            for _ in range(2):
                e = ctypes.c_void_p()
                rc = hip.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE)
                if rc != 0:
                    raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")
                pair.append(e)
            self.pairs.append(tuple(pair))

    def arm(self, i: int) -> None:
        from paper_2609_36760_amd import _binding as mb
        mb.mla_time_next_decode_launch(self.pairs[i][0].value, self.pairs[i][1].value)

    def elapsed_ms(self, i: int) -> float:
        f = self._c.c_float()
        rc = self._hip.hipEventElapsedTime(self._c.byref(f), self.pairs[i][0], self.pairs[i][1])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return f.value

    def __del__(self):
        for pair in getattr(self, "pairs", []):
            for e in pair:
                self._hip.hipEventDestroy(e)


def algorithmic_bytes(run) -> int:
    """HBM bytes one decode launch must move: every attended key once, queries,
    and the split partials (fp16 normalized latent, fp32 max and sum) or the
    output."""
    keys = run.key_bytes()
    q = run.B * run.s_q * run.H * (512 + 64) * 2
    rows = run.B * run.s_q * run.H
    if run.split_tokens:
        parts = run.num_splits * run.s_q * run.H * (512 * 2 + 2 * 4)   # fp16 latent, fp32 max and sum
        return keys + q + parts
    return keys + q + rows * 512 * 2


class ClockSampler:
    """Samples the GPU's graphics clock (torch.cuda.clock_rate, MHz) and its
    average socket power (torch.cuda.power_draw, amdsmi's
    average_socket_power, W) from a host thread.  amdsmi refreshes these
    about once a second, so the figures mean something only over a run of
    seconds: ``sustained`` runs the step back to back for that long and keeps
    the samples after the first third (the clock's ramp from idle)."""

    def __init__(self, period_s: float = 0.02):
        import threading
        self.samples, self.power, self._stop, self.period = [], [], threading.Event(), period_s
        self._t = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        import torch
        while not self._stop.is_set():
            try:
                self.samples.append(float(torch.cuda.clock_rate()))
            except Exception:
                return
            try:
                self.power.append(float(torch.cuda.power_draw()))
            except Exception:
                pass
            time.sleep(self.period)

    def __enter__(self):
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join()

    def summary(self, seconds):
        if not self.samples:
            return None
        a = np.asarray(self.samples[len(self.samples) // 3:])
        out = {"median_mhz": float(np.median(a)), "min_mhz": float(a.min()), "max_mhz": float(a.max()),
               "samples": int(a.size), "seconds": seconds,
               "source": "amdsmi, sampled every 20 ms while the step runs back to back; first third dropped"}
        p = np.asarray(self.power[len(self.power) // 3:])
        if p.size and p.max() > 0:
            out["socket_power_w"] = {"median": float(np.median(p)), "max": float(p.max())}
        return out


def sustained(one_step, seconds=1.5, burst=50):
    """Clock and socket power while ``one_step`` runs back to back for
    ``seconds`` (bursts of ``burst`` steps, synchronized between bursts)."""
    import torch
    with ClockSampler() as smp:
        t0, i = time.perf_counter(), 0
        while time.perf_counter() - t0 < seconds:
            for _ in range(burst):
                one_step(i)
                i += 1
            torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    res = smp.summary(round(wall, 2))
    if res is not None:
        res["ms_per_step"] = wall * 1e3 / i
    return res


def stats_of(a):
    a = np.asarray(a, np.float64)
    return {"mean": float(a.mean()), "median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90)), "n": int(a.size)}


def make_run(name, kind, token_cache=None, protect=None, split_tokens=None, meta="fp16", layer=0,
             device_tokens=False):
    import torch

    from paper_2609_36760_amd import synthetic as syn
    from paper_2609_36760_amd.runner import DecodeRun
    t0 = time.perf_counter()
    run = DecodeRun(syn.WORKLOADS[name], layer=layer, kind=kind, token_cache=token_cache, protect=protect,
                    split_tokens=split_tokens, meta=meta, device_tokens=device_tokens)
    torch.cuda.synchronize()
    log(f"[{name} {kind}] setup {time.perf_counter() - t0:.1f}s, cache {run.cache.numel() / 1e6:.1f} MB")
    return run


def time_workload(name, kind, steps, warmup, layers, token_cache=None, protect=None, split_tokens=None,
                  meta="fp16", layer=0, device_tokens=False, run=None, clock=False):
    """Time ``steps`` steps after ``warmup`` untimed ones, cycling ``layers``
    resident caches; returns the step and per-launch kernel figures."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    own = run is None
    if own:
        run = make_run(name, kind, token_cache, protect, split_tokens, meta, layer, device_tokens)
    protect = run.protect
    caches = [run.cache] + [run.cache.clone() for _ in range(layers - 1)]
    prots = [None] * layers if protect is None else [run.prot] + [run.prot.clone() for _ in range(layers - 1)]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    fused = mb.mla_lowbit_append_decode_attn if kind == "lowbit" else mb.mla_bf16_append_decode_attn

    def one_step(i, ev=None):
        cache, prot = caches[i % layers], prots[i % layers]
        if protect is None:
            # the append runs inside the decode launch (the same cache bytes and
            # outputs as the writer launch followed by the decode)
            if ev is not None:
                ev.arm(i - warmup)
            fused(run.fmt, run.new_c, run.new_k, run.new_slots, run.q_lat, run.q_rope, cache, run.num_pages,
                  run.block_table, run.seq_lens, run.s_q, run.H, run.tau, split_tokens=run.split_tokens,
                  split_indptr=run.split_indptr, num_splits=run.num_splits, out=run.out, lse=run.lse,
                  part_m=run.part_m, part_s=run.part_s, part_o=run.part_o, stream=sh)
        else:
            # under protection too: the new tokens' packed bytes and bf16 rows are
            # written inside the decode launch
            if ev is not None:
                ev.arm(i - warmup)
            mb.mla_lowbit_append_decode_attn_protected(
                run.fmt, protect, run.new_c, run.new_k, run.new_slots, run.q_lat, run.q_rope, cache, run.num_pages,
                run.block_table, run.seq_lens, run.s_q, run.H, run.tau, prot, run.num_prot, run.prot_slot,
                split_tokens=run.split_tokens, split_indptr=run.split_indptr, num_splits=run.num_splits,
                out=run.out, lse=run.lse, part_m=run.part_m, part_s=run.part_s, part_o=run.part_o, stream=sh)
        if run.split_tokens:
            mb.mla_splitkv_combine(run.part_m, run.part_s, run.part_o, run.split_indptr, run.num_splits, run.B,
                                   run.s_q, run.H, run.out, run.lse, stream=sh)

    for i in range(warmup):
        one_step(i)
    evs = TimingEvents(steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(warmup, warmup + steps):
        one_step(i, evs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern = [evs.elapsed_ms(k) for k in range(steps)]
    kern_ms = float(np.mean(kern))
    ms_step = wall * 1e3 / steps
    flops = run.flops()
    nbytes = algorithmic_bytes(run)
    res = {
        "workload": name, "kind": kind, "ms_per_step": ms_step,
        "decode_tokens_per_s": run.B * run.s_q / (ms_step * 1e-3),
        "kv_tokens_per_s": float(run.lens.sum()) / (ms_step * 1e-3),
        "decode_kernel_ms": kern_ms,
        "decode_kernel_ms_stats": stats_of(kern),
        "decode_kernel_tflops": flops / (kern_ms * 1e-3) / 1e12,
        "decode_kernel_gbs": nbytes / (kern_ms * 1e-3) / 1e9,
        "flops_per_launch": flops, "bytes_per_launch": nbytes,
        "splits": run.num_splits, "split_tokens": run.split_tokens, "layers_cycled": layers,
    }
    res["mfma_frac"] = res["decode_kernel_tflops"] / PEAK_BF16_TFLOPS
    res["hbm_frac"] = res["decode_kernel_gbs"] / PEAK_HBM_GBS
    if clock:
        res["gpu_clock"] = sustained(lambda i: one_step(warmup + steps + i))
    if protect is not None:
        res["protect"] = {"sink": protect.sink, "recent": protect.recent}
    tag = ("" if protect is None else " protected") + ("" if meta == "fp16" else f" {meta} metadata")
    log(f"[{name} {kind}{tag}] {ms_step * 1e3:.1f} us/step, decode kernel {kern_ms * 1e3:.1f} us "
        f"(median {res['decode_kernel_ms_stats']['median'] * 1e3:.1f}) = "
        f"{res['decode_kernel_tflops']:.1f} TFLOP/s ({100 * res['mfma_frac']:.1f}% MFMA), "
        f"{res['decode_kernel_gbs']:.0f} GB/s ({100 * res['hbm_frac']:.1f}% HBM)"
        + (f", sustained clock {res['gpu_clock']}" if clock else ""))
    del caches, prots
    if own:
        del run
        torch.cuda.empty_cache()
    return res


def latency_protocol(runs, runs_per=2, rounds=2, samples=30, flush_bytes=1 << 30):
    """The paper's kernel-latency protocol (Appendix F.1): attention + combine
    replayed from a captured HIP graph, the L2 and last-level caches flushed
    (a 1 GiB write) before every sample, HIP events around the replay,
    ``runs_per`` runs x ``rounds`` rounds x ``samples`` samples with the
    kinds' order alternating between rounds.  ``runs``: {label: DecodeRun}."""
    import torch
    flush = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda")
    graphs, mode = {}, "graph"
    for label, run in runs.items():
        run.attend()                                 # warm, outside the capture
        torch.cuda.synchronize()
        try:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run.attend()
            graphs[label] = g.replay
        except Exception as e:                       # the capture failed: time eager launches
            log(f"graph capture of {label} failed ({e}); timing eager launches")
            graphs[label] = run.attend
            mode = "eager"
    torch.cuda.synchronize()
    lat = {label: [] for label in runs}
    labels = list(runs)
    stream = torch.cuda.current_stream()
    for r in range(runs_per):
        for rd in range(rounds):
            order = labels if (r + rd) % 2 == 0 else labels[::-1]
            for label in order:
                for i in range(samples):
                    flush.fill_((r * 7 + rd * 3 + i) & 0xFF)
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    graphs[label]()
                    e1.record(stream)
                    torch.cuda.synchronize()
                    lat[label].append(e0.elapsed_time(e1) * 1e3)
    del flush
    torch.cuda.empty_cache()
    out = {"replay": mode, "runs": runs_per, "rounds": rounds, "samples_per_round": samples,
           "flush_bytes": flush_bytes, "unit": "us"}
    for label, v in lat.items():
        out[label] = stats_of(v)
        log(f"[protocol {label}] {mode}: mean {out[label]['mean']:.1f} us, median {out[label]['median']:.1f}, "
            f"p10 {out[label]['p10']:.1f}, p90 {out[label]['p90']:.1f}")
    return out


def environment():
    import platform

    import torch
    rocm = None
    try:
        rocm = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        pass
    props = torch.cuda.get_device_properties(0)
    return {"device": props.name, "gcn_arch": getattr(props, "gcnArchName", None),
            "compute_units": props.multi_processor_count, "rocm": rocm, "torch_hip": torch.version.hip,
            "host_cpus": os.cpu_count(), "python": platform.python_version()}


def cpu_baseline(budget_s: float = 15.0):
    """The oracle, as it stands, on whole sequences of the headline workload
    (quantize and pack of every cached token, then fp64 attention of all
    heads), for about ``budget_s`` seconds."""
    from oracle import attention as at
    from oracle import paged_cache as pc
    from paper_2609_36760_amd import synthetic as syn
    w = syn.WORKLOADS[MAIN]
    fmt = pc.CacheFormat(c_bits=w.layers[0][0], r_bits=w.layers[0][1])
    lens = syn.seq_lens(w)
    done, spent = 0, 0.0
    while done < w.B and spent < budget_s:
        b = done
        c, k = syn.sequence_tokens(w, 0, b, int(lens[b]))
        ql, qr = syn.queries(w, 0, batch=[b])
        ts = time.perf_counter()
        c_hat, kr_hat = pc.encode_sequence_dense(fmt, c, k)
        at.decode_sequence(ql[0], qr[0], c_hat, kr_hat, w.tau)
        spent += time.perf_counter() - ts
        done += 1
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        blas = 1
    return {"value": done * w.s_q / spent, "unit": "tokens/s", "cores": blas, "host_cpus": os.cpu_count(),
            "kind": "oracle",
            "sample": f"{done} of {w.B} sequences of {MAIN} (32768 tokens, 128 heads each): fp32 quantize and "
                      f"pack of every cached token and fp64 attention of all heads; oracle time {spent:.1f}s on "
                      f"{blas} BLAS threads of {os.cpu_count()} host CPUs (input generation excluded)"}


ORACLE_CONFIGS = (("tiny_b1_h16_256", 0), ("dsv3_b32_h128_4k_c4r4", 0), ("int2_b64_h128_32k_c2r4", 0),
                  ("splitkv_b8_h128_128k_c4r4", 0), ("ragged_b96_h128_sq2_mixed", 0),
                  ("ragged_b96_h128_sq2_mixed", 1), (MAIN, 0))


def cpu_baseline_configs():
    """The CPU baseline over every full-size configuration in full: the oracle,
    as it stands, on every sequence -- (i) the fp32 quantize and pack of every
    cached token (Appendix C.4), (ii) the dequantization and fp64 attention of
    every row (Sec. 2.1), through per-split partials and their global merge
    (Appendix C.5) where the configuration splits its keys.  Wall time per
    configuration on the host's cores; inputs drawn outside the timed parts."""
    from oracle import attention as at
    from oracle import paged_cache as pc
    from paper_2609_36760_amd import synthetic as syn
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        blas = 1
    rows = []
    for name, layer in ORACLE_CONFIGS:
        w = syn.WORKLOADS[name]
        fmt = pc.CacheFormat(c_bits=w.layers[layer][0], r_bits=w.layers[layer][1])
        lens = syn.seq_lens(w)
        t_pack = t_attn = 0.0
        for b in range(w.B):
            L = int(lens[b])
            c, k = syn.sequence_tokens(w, layer, b, L)
            ql, qr = syn.queries(w, layer, batch=[b])
            t0 = time.perf_counter()
            blocks = pc.encode_tokens(fmt, c, k)
            t1 = time.perf_counter()
            c_hat, kr_hat = pc.decode_blocks(fmt, blocks)
            if w.split_tokens:
                R = w.s_q * w.H
                bounds = [(a, min(a + w.split_tokens, L)) for a in range(0, L, w.split_tokens)]
                m, s_, o = at.chunk_partials(at.bf16_bits_to_f64(ql[0]).reshape(R, -1),
                                             at.bf16_bits_to_f64(qr[0]).reshape(R, -1), c_hat, kr_hat, w.tau,
                                             at.decode_limits(L, w.s_q, w.H), bounds)
                at.merge(m, s_, o)
            else:
                at.decode_sequence(ql[0], qr[0], c_hat, kr_hat, w.tau)
            t2 = time.perf_counter()
            t_pack += t1 - t0
            t_attn += t2 - t1
        tokens = int(lens.sum())
        rows.append({"workload": name, "layer": layer, "sequences": int(w.B), "cached_tokens": tokens,
                     "rows": int(w.B * w.s_q * w.H), "splits": w.split_tokens or None,
                     "quantize_pack_s": round(t_pack, 2), "dequant_attention_merge_s": round(t_attn, 2),
                     "decode_tokens_per_s": round(w.B * w.s_q / (t_pack + t_attn), 3)})
        print(f"[oracle {name} layer {layer}] pack {t_pack:.1f} s, attention {t_attn:.1f} s "
              f"({tokens} tokens)", file=sys.stderr, flush=True)
    return {"kind": "oracle", "cores": blas, "host_cpus": os.cpu_count(), "configs": rows}


def measured_traffic(workload: str):
    """HBM bytes per launch of the low-bit decode kernel on ``workload`` from
    the recorded FETCH_SIZE / WRITE_SIZE counter runs, each scaled by what the
    same counter read for a plain 256 MiB copy; None when there is no record
    for the workload or the kernel sources changed since it was taken."""
    import hashlib
    pkg = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2609_36760_amd")
    try:
        recs = json.load(open(os.path.join(pkg, "measured_traffic.json")))["records"]
    except (OSError, KeyError, ValueError):
        return None
    for rec in recs:
        if rec.get("workload") != workload:
            continue
        try:
            h = hashlib.sha256()
            for f in rec["kernel_sources"]:
                h.update(open(os.path.join(pkg, f), "rb").read())
        except (OSError, KeyError):
            return None
        if h.hexdigest() != rec["kernel_sources_sha256"]:
            return None
        kib = rec["copy_bytes"] / 1024.0
        fetch = rec["fetch_kib_per_dispatch"] * kib / rec["copy_fetch_kib"] * 1024.0
        write = rec["write_kib_per_dispatch"] * kib / rec["copy_write_kib"] * 1024.0
        return fetch + write
    return None


# The paper's attention latency table (Appendix F.1): 16 heads, one query token,
# C4R4 with sink 4 / recent 128 against a BF16 cache, on its own (unnamed
# NVIDIA) GPU, microseconds.  Context only.
PAPER_GRID_US = {
    (8, 1024): (25.69, 23.78), (8, 4096): (51.43, 53.63), (8, 8192): (82.50, 85.35),
    (8, 16384): (147.34, 149.79), (8, 32768): (281.44, 281.99), (8, 65536): (542.14, 540.61),
    (8, 131072): (1067.24, 1062.32), (8, 262144): (2122.10, 2113.33), (8, 524288): (4234.79, 4214.84),
    (8, 1048576): (8440.05, 8418.63),
    (32, 1024): (55.50, 56.97), (32, 4096): (156.82, 155.54), (32, 8192): (287.58, 283.46),
    (32, 16384): (548.73, 547.20), (32, 32768): (1072.93, 1067.28), (32, 65536): (2133.71, 2124.10),
    (32, 131072): (4236.96, 4225.35), (32, 262144): (8449.30, 8426.35), (32, 524288): (16880.19, 16827.11),
    (32, 1048576): (33701.48, 33609.17),
}


def grid_split(B: int, n_list: int, target: int = 1024) -> int:
    """Key split (tokens) giving about `target` work items over B sequences of
    n_list 32-key list tiles (at least 64 tokens per split)."""
    per = max(2, -(-B * n_list // target))
    return 32 * per


CONFIG_SHAPES = (
    # (workload, cache layer, label)
    ("int2_b64_h128_32k_c2r4", 0, "C2R4, 64 x 32K"),
    ("splitkv_b8_h128_128k_c4r4", 0, "C4R4, 8 x 128K, 64 splits of 2048"),
    ("ragged_b96_h128_sq2_mixed", 0, "C4R4 layer, 96 ragged 1K-128K, s_q 2, 2 tokens appended"),
    ("ragged_b96_h128_sq2_mixed", 1, "C2R4 layer, 96 ragged 1K-128K, s_q 2, 2 tokens appended"),
)


def config_report(args):
    """The full-size correctness configurations timed like the bench workload
    (append inside the decode launch, then the combine; one resident cache),
    low-bit and BF16 cache, with the roofline that binds each: a kernel is
    MFMA-bound when its algorithmic intensity (flop per HBM byte) exceeds the
    ridge 2500 TFLOP/s / 8 TB/s = 312.5 flop/B, else HBM-bound."""
    ridge = PEAK_BF16_TFLOPS / (PEAK_HBM_GBS / 1e3)
    rows = []
    for name, layer, label in CONFIG_SHAPES:
        res = {"workload": name, "layer": layer, "label": label}
        for kind in ("lowbit", "bf16"):
            r = time_workload(name, kind, args.config_steps, args.config_warmup, 1, layer=layer, device_tokens=True)
            inten = r["flops_per_launch"] / r["bytes_per_launch"]
            bound = "mfma" if inten > ridge else "hbm"
            r["intensity_flop_per_byte"] = inten
            r["bound"] = bound
            r["frac_of_binding_roofline"] = r["mfma_frac"] if bound == "mfma" else r["hbm_frac"]
            res[kind] = r
        res["speedup_vs_bf16"] = res["bf16"]["ms_per_step"] / res["lowbit"]["ms_per_step"]
        rows.append(res)
    print(json.dumps({"metric": METRIC, "report": "configs", "ridge_flop_per_byte": ridge, "configs": rows}),
          flush=True)


def paper_grid(args):
    """Attention latency over the paper's grid: decode + combine, L2 flushed
    (a 512 MiB write) before every sample, HIP events on the launch stream."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd import synthetic as syn
    from paper_2609_36760_amd.runner import DecodeRun
    contexts = [int(x) for x in args.grid_contexts.split(",")]
    batches = [int(x) for x in args.grid_batches.split(",")]
    pol = mb.protect_policy(4, 128)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    rows = []
    for B in batches:
        for N in contexts:
            rec = {"batch": B, "context": N}
            for label, kind, protect in (("c4r4", "lowbit", pol), ("bf16", "bf16", None)):
                n_list = (-(-(N - 128) // 32) + 5) if protect is not None else -(-N // 32)
                split = grid_split(B, n_list)
                w = syn.Workload(f"paper_h16_b{B}_{N}", 60, B=B, H=16, s_q=1, context=N)
                t0 = time.perf_counter()
                run = DecodeRun(w, kind=kind, protect=protect, split_tokens=split, device_tokens=True)
                run.append_new_tokens()
                torch.cuda.synchronize()
                setup = time.perf_counter() - t0
                lat = []
                for i in range(args.grid_warmup + args.grid_samples):
                    flush.fill_(i & 0xFF)
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    run.attend()
                    e1.record(stream)
                    torch.cuda.synchronize()
                    if i >= args.grid_warmup:
                        lat.append(e0.elapsed_time(e1) * 1e3)
                us = float(np.mean(lat))
                nbytes = algorithmic_bytes(run)
                rec[label] = {"us": us, "us_min": float(np.min(lat)), "splits": run.num_splits,
                              "split_tokens": split, "bytes": nbytes, "gbs": nbytes / (us * 1e-6) / 1e9,
                              "hbm_frac": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}
                log(f"[grid B={B} N={N} {label}] setup {setup:.1f}s, {us:.1f} us (min {np.min(lat):.1f}), "
                    f"{run.num_splits} splits of {split}, {rec[label]['gbs']:.0f} GB/s")
                del run
                torch.cuda.empty_cache()
            rec["speedup_vs_bf16"] = rec["bf16"]["us"] / rec["c4r4"]["us"]
            paper = PAPER_GRID_US.get((B, N))
            rec["paper_us"] = None if paper is None else {"bf16": paper[0], "c4r4": paper[1]}
            rows.append(rec)
            print(json.dumps(rec), flush=True)
    print(json.dumps({"metric": "attention latency, 16 heads, C4R4 sink4/local128 vs BF16",
                      "unit": "us", "grid": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300, help="timed steps of the headline workload")
    ap.add_argument("--warmup", type=int, default=300,
                    help="untimed steps first: the clock ramps up from idle over the first tens of milliseconds")
    ap.add_argument("--small-steps", type=int, default=300, help="timed steps of the 32 x 4096 workload")
    ap.add_argument("--small-warmup", type=int, default=300)
    ap.add_argument("--no-sustain", action="store_true",
                    help="skip the 1.5 s back-to-back runs that measure the sustained clock and power")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-protocol", action="store_true", help="skip the paper's sampling protocol")
    ap.add_argument("--kinds", default="lowbit,bf16,small,protected,paper",
                    help="what to time besides the headline: bf16 (the BF16 cache at both shapes), small (the 32 x "
                         "4096 workload), protected (4 sink / 128 recent bf16 protection at 32 x 4096), paper (the "
                         "paper's metadata storage at 32 x 4096); 'lowbit' alone times only the headline")
    ap.add_argument("--protect-split", type=int, default=0,
                    help="key split of the protected step (0: as many splits per sequence as the unprotected plan)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="first copy a 256 MiB buffer once (reference for HBM traffic counters)")
    ap.add_argument("--paper-grid", action="store_true",
                    help="instead of the step benchmark: the paper's 16-head attention latency grid")
    ap.add_argument("--oracle-configs", action="store_true",
                    help="time the CPU oracle on every full-size configuration in full (no GPU use) and exit")
    ap.add_argument("--configs", action="store_true",
                    help="report the full-size correctness configurations instead (one JSON line)")
    ap.add_argument("--config-steps", type=int, default=100)
    ap.add_argument("--config-warmup", type=int, default=100)
    ap.add_argument("--grid-batches", default="8,32")
    ap.add_argument("--grid-contexts", default="1024,4096,8192,16384,32768,65536,131072,262144,524288,1048576")
    ap.add_argument("--grid-samples", type=int, default=30)
    ap.add_argument("--grid-warmup", type=int, default=5)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no multi-GPU path; "
              "the per-GPU kernel is the whole workload.", file=sys.stderr)
        sys.exit(2)
    if args.oracle_configs:
        print(json.dumps({"oracle_configs": cpu_baseline_configs()}), flush=True)
        return
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    if args.paper_grid:
        paper_grid(args)
        return
    if args.configs:
        config_report(args)
        return
    if args.calib_copy:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)                      # reads and writes exactly 256 MiB
        torch.cuda.synchronize()
        del src, dst
    kinds = args.kinds.split(",")
    env = environment()
    tc = {}
    run_lb = make_run(MAIN, "lowbit", token_cache=tc)
    main_lb = time_workload(MAIN, "lowbit", args.steps, args.warmup, LAYERS[MAIN], run=run_lb,
                            clock=not args.no_sustain)
    extra = {}
    main_bf = None
    run_bf = None
    if "bf16" in kinds:
        run_bf = make_run(MAIN, "bf16", token_cache=tc)
        main_bf = time_workload(MAIN, "bf16", args.steps, args.warmup, LAYERS[MAIN], run=run_bf,
                                clock=not args.no_sustain)
    del tc
    if not args.no_protocol:
        runs = {"c4r4": run_lb} if run_bf is None else {"c4r4": run_lb, "bf16": run_bf}
        extra["latency_protocol"] = latency_protocol(runs)
        if "bf16" in runs:
            extra["latency_protocol"]["speedup_vs_bf16_median"] = (extra["latency_protocol"]["bf16"]["median"] /
                                                                  extra["latency_protocol"]["c4r4"]["median"])
    del run_lb, run_bf
    torch.cuda.empty_cache()

    if "small" in kinds:
        sm = time_workload(SMALL, "lowbit", args.small_steps, args.small_warmup, LAYERS[SMALL])
        entry = {"c4r4": sm}
        if "bf16" in kinds:
            sb = time_workload(SMALL, "bf16", args.small_steps, args.small_warmup, LAYERS[SMALL])
            entry["bf16"] = sb
            entry["speedup_vs_bf16"] = sb["ms_per_step"] / sm["ms_per_step"]
        entry["traffic"] = measured_traffic(SMALL)
        extra[SMALL] = entry
    if "protected" in kinds:
        from paper_2609_36760_amd import _binding as mb
        from paper_2609_36760_amd import synthetic as syn
        pol = mb.protect_policy(4, 128)

        def protect_split(name):
            # as many key splits per sequence as the unprotected plan: the tile list
            # (packed tiles + protected rows) is one tile longer than the sequence
            w = syn.WORKLOADS[name]
            L = w.context
            n_list = -(-(L - pol.recent) // 32) - pol.sink // 32 + -(-(pol.sink + pol.recent) // 32)
            return 32 * -(-n_list // -(-L // w.split_tokens))

        pr = time_workload(SMALL, "lowbit", args.small_steps, args.small_warmup, LAYERS[SMALL], protect=pol,
                           split_tokens=args.protect_split or protect_split(SMALL))
        pr["step_vs_unprotected"] = (extra[SMALL]["c4r4"]["ms_per_step"] / pr["ms_per_step"]
                                     if SMALL in extra else None)
        extra["protected_sink4_recent128_" + SMALL] = pr
        # the paper's policy at the headline shape (its efficiency runs all use it)
        pm = time_workload(MAIN, "lowbit", args.steps, args.warmup, LAYERS[MAIN], protect=pol,
                           split_tokens=protect_split(MAIN), device_tokens=True)
        pm["step_vs_unprotected"] = main_lb["ms_per_step"] / pm["ms_per_step"]
        extra["protected_sink4_recent128_" + MAIN] = pm
    if "paper" in kinds:
        pp = time_workload(SMALL, "lowbit", args.small_steps, args.small_warmup, LAYERS[SMALL], meta="paper")
        pp["cache_bytes_per_token"] = 320
        extra["paper_storage_c4r4_" + SMALL] = pp
    cpu = None if args.no_cpu else cpu_baseline()

    line = {
        "metric": METRIC,
        "value": main_lb["decode_tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": main_lb["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp16",
        "dtype_detail": "INT4 codes dequantized to fp16 MFMA operands, fp32 accumulation; bf16 queries and outputs",
        "data": "synthetic",
        "config": {"workload": MAIN, "batch": 64, "heads": 128, "context": 32768, "s_q": 1,
                   "cache": "INT4 content + INT4 RoPE key, group 64, fp16 scale/zero",
                   "split_tokens": main_lb["split_tokens"], "layers_cycled": LAYERS[MAIN]},
        "roofline": {"bound": "mfma", "achieved": main_lb["decode_kernel_tflops"], "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": main_lb["mfma_frac"], "traffic": measured_traffic(MAIN),
                     "algorithmic_bytes": main_lb["bytes_per_launch"],
                     "algorithmic_flops": main_lb["flops_per_launch"],
                     "kernel_ms": main_lb["decode_kernel_ms_stats"]},
        "gpu_clock": main_lb.get("gpu_clock"),
        "hbm_gbs": main_lb["decode_kernel_gbs"], "hbm_frac": main_lb["hbm_frac"],
        "bf16_cache": None if main_bf is None else {
            "value": main_bf["decode_tokens_per_s"], "ms_per_step": main_bf["ms_per_step"],
            "decode_kernel_ms": main_bf["decode_kernel_ms"], "kernel_ms": main_bf["decode_kernel_ms_stats"],
            "hbm_gbs": main_bf["decode_kernel_gbs"], "hbm_frac": main_bf["hbm_frac"],
            "mfma_frac": main_bf["mfma_frac"], "bound": "hbm", "gpu_clock": main_bf.get("gpu_clock")},
        "speedup_vs_bf16": None if main_bf is None else main_bf["ms_per_step"] / main_lb["ms_per_step"],
        "cpu_baseline": cpu,
        "environment": env,
        "context": {"paper_kv_compression_128k": 3.59, "paper_serving_speedup_vs_bf16": 5.168,
                    "paper_hardware": "unnamed NVIDIA GPUs (one for kernels, eight for serving)"},
    }
    line.update(extra)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

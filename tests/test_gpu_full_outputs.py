"""Every output of every full-size configuration against the oracle (GPU;
about a minute and a half, most of it the oracle on 16 host cores).

The default suite checks sampled sequences and heads at full size
(``test_gpu_decode.py``).  This test checks all B x s_q x H x 512 outputs and
every lse of each full-size configuration and of the 64 x 32768 shape, for the
low-bit cache and, at the two 128-head benchmark shapes, the BF16 cache: the
step the benchmark times (the step's tokens appended inside the decode launch,
then the combine), against the oracle's attention (Sec. 2.1, eq. mla_compact)
over the values the stored bytes hold, with the global rule and bounds of
``gpu_support`` applied per configuration.  The oracle runs per sequence in
16 worker processes (started fresh, no GPU use); each packs the sequence's
tokens (Appendix C.4, "Affine group quantization"), checks the packing
against a digest of the GPU's pages (the BF16 cache: its rows) -- every
byte of every cache, 10.8M low-bit tokens in all -- decodes it and returns
its sequence's statistics.

Over all outputs, some configurations break the max rule in a few rows:
outlier channels (10x) whose output is tens of times the RMS, in rows whose
weight sits on one or two keys.  There the 16-bit operands of the datapath
(fp16 reconstructed latents and weights, fp16 split partials; the BF16
kernel: bf16 weights) move the output by more than 2e-2 of the RMS, or leave
an fp16 partial on a bf16 rounding tie.  Every such row is then checked
against a model of the kernel's own rounding instead
(``test_precision_budget._emulate`` with the rows of the row's wave: the
same key ranges, 32-key tiles, fp16/bf16 roundings and wave-uniform lazy
reference, fp64 otherwise):
  * each split partial of the GPU (fp16 normalized sum) equals the model's
    unrounded partial up to its own fp16 rounding plus 2^-14 of the row's
    largest element; its maximum within 1e-4 and its weight sum within a
    relative 2^-12;
  * the output equals the exact combine of the GPU's own partials, rounded to
    bf16 (within a relative 2^-17 of a rounding tie).
Every other rule is asserted against the oracle, and the max rule is then
reported as an expected failure, with the count of the rows that break it.
"""
import hashlib
import multiprocessing as mp
import time

import numpy as np
import pytest

from gpu_support import MAX_TOL, AttnStats, bf16_bits_to_f64, compare_sequence, gpu_pages, half_ulp_bf16, oracle_format
from oracle import paged_cache as pc
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

CONFIGS = [
    # (workload, layer, kind)
    ("tiny_b1_h16_256", 0, "lowbit"),
    ("dsv3_b32_h128_4k_c4r4", 0, "lowbit"),
    ("dsv3_b32_h128_4k_c4r4", 0, "bf16"),
    ("int2_b64_h128_32k_c2r4", 0, "lowbit"),
    ("splitkv_b8_h128_128k_c4r4", 0, "lowbit"),
    ("ragged_b96_h128_sq2_mixed", 0, "lowbit"),
    ("ragged_b96_h128_sq2_mixed", 1, "lowbit"),
    ("c4r4_b64_h128_32k", 0, "lowbit"),
    ("c4r4_b64_h128_32k", 0, "bf16"),
]


def _digest(blocks):
    h = hashlib.sha256()
    for blk in blocks:
        h.update(np.ascontiguousarray(blk).tobytes())
    return h.hexdigest()


def _values(name, layer, kind, b, L, c_bits, r_bits, meta, digest):
    """The oracle's values of sequence b (fp64) and whether the GPU bytes'
    digest matches the oracle's packing (BF16: the rows themselves)."""
    w = syn.WORKLOADS[name]
    c_bits16, k_bits16 = syn.sequence_tokens(w, layer, b, L)
    if kind == "bf16":
        ok = digest == _digest([np.concatenate([c_bits16, k_bits16], axis=1)])
        return ok, bf16_bits_to_f64(c_bits16), bf16_bits_to_f64(k_bits16)
    fmt = pc.CacheFormat(c_bits=c_bits, r_bits=r_bits, meta=meta)
    blocks = pc.encode_tokens(fmt, c_bits16, k_bits16)
    c, k = (x.astype(np.float64) for x in pc.decode_blocks(fmt, blocks))
    return digest == _digest(blocks), c, k


def oracle_sequence(job):
    """Worker: the oracle's attention of sequence b compared with the GPU's
    outputs; returns the statistics and each row's largest max-rule excess
    (|gpu - oracle| less half a bf16 ulp of the oracle value)."""
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)                    # 16 workers on 16 host cores
    name, layer, kind, b, L, c_bits, r_bits, meta, digest, got_out, got_lse, tau = job
    w = syn.WORKLOADS[name]
    ok, c, k = _values(name, layer, kind, b, L, c_bits, r_bits, meta, digest)
    ql, qr = syn.queries(w, layer, batch=[b])
    stats = AttnStats()
    want = compare_sequence(stats, got_out, got_lse, ql[0], qr[0], c, k, tau, w.s_q)
    excess = np.maximum(np.abs(bf16_bits_to_f64(got_out) - want) - half_ulp_bf16(want), 0.0).max(axis=-1)
    return b, ok, stats, excess


def model_rows(job):
    """Worker: the rounding model's unrounded split partials of the 32 rows of
    one wave (query token i, heads ``heads``) of sequence b."""
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)
    import test_precision_budget as tp
    from oracle import attention as at
    name, layer, kind, b, L, c_bits, r_bits, meta, digest, tau, split, i, heads = job
    w = syn.WORKLOADS[name]
    ok, c, k = _values(name, layer, kind, b, L, c_bits, r_bits, meta, digest)
    ql, qr = syn.queries(w, layer, batch=[b])
    kv, p = (tp._ident, tp._rnd_bf16) if kind == "bf16" else (tp._rnd_f16, tp._rnd_f16)
    a = at.bf16_bits_to_f64(ql[0][i, heads])
    r = at.bf16_bits_to_f64(qr[0][i, heads])
    parts = tp._emulate(a, r, c, k, tau, w.s_q, kv, p, split=split, groups=np.zeros(len(heads), int),
                        lim=np.full(len(heads), L - w.s_q + 1 + i), partials=True,
                        p_format="bf16" if kind == "bf16" else "f16")
    return b, i, ok, parts


def _check_modelled(name, run, out, b, i, heads, parts):
    """The modelled wave's GPU partials against the model's, and its outputs
    against the exact combine of those partials; returns the largest partial
    excess (beyond its fp16 rounding) over the row's largest element."""
    H, R = run.H, run.s_q * run.H
    j0, j1 = int(run.split_indptr_host[b]), int(run.split_indptr_host[b + 1])
    assert j1 - j0 == len(parts)
    rows = i * H + np.asarray(heads)
    po = run.part_o.view(run.num_splits, R, 512)[j0:j1].cpu().numpy()[:, rows].astype(np.float64)
    pm = run.part_m.view(run.num_splits, R)[j0:j1].cpu().numpy()[:, rows].astype(np.float64)
    ps = run.part_s.view(run.num_splits, R)[j0:j1].cpu().numpy()[:, rows].astype(np.float64)
    worst = 0.0
    for j, (m, s, u, tol_u, tol_s) in enumerate(parts):
        vis = s > 0
        half16 = np.exp2(np.floor(np.log2(np.maximum(np.abs(u), 2.0 ** -14))) - 11)
        top = np.abs(u).max(axis=1, keepdims=True)
        ex = np.maximum(np.abs(po[j] - u) - half16 - tol_u, 0.0)
        assert np.all(ex[vis] <= 2.0 ** -15 * top[vis] + 2.0 ** -25), \
            f"{name} seq {b} token {i} split {j}: partial {float((ex / np.maximum(top, 1e-30)).max()):.2e} " \
            f"of the row's largest element from the rounding model"
        assert np.all(np.abs(pm[j][vis] - m[vis]) <= 1e-4), f"{name} seq {b} token {i} split {j}: partial maximum"
        assert np.all(np.abs(ps[j][vis] - s[vis]) <= tol_s[vis] + 2.0 ** -15 * s[vis]), \
            f"{name} seq {b} token {i} split {j}: weight sum"
        worst = max(worst, float((ex[vis] / top[vis]).max(initial=0.0)))
    M = pm.max(axis=0)
    W = np.exp(pm - M) * ps                                   # [splits, rows]
    comb = (W[..., None] * po).sum(axis=0) / W.sum(axis=0)[:, None]
    g = bf16_bits_to_f64(out[b][i, heads])
    assert np.all(np.abs(g - comb) <= half_ulp_bf16(comb) + 2.0 ** -17 * np.abs(comb)), \
        f"{name} seq {b} token {i}: output is not the bf16 rounding of the combined partials"
    return worst


@pytest.mark.parametrize("config", CONFIGS, ids=[f"{n}-L{l}-{k}" for n, l, k in CONFIGS])
def test_full_outputs(config):
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    name, layer, kind = config
    t0 = time.perf_counter()
    run = DecodeRun(syn.WORKLOADS[name], layer=layer, kind=kind)
    run.fused_step()
    torch.cuda.synchronize()
    out, lse = run.out.cpu().numpy(), run.lse.cpu().numpy()
    lens = [int(x) for x in run.lens]
    jobs = []
    for b, L in enumerate(lens):
        pages = gpu_pages(run, b)
        if kind == "bf16":
            digest = _digest([pages.view(np.uint16).reshape(-1, 576)[:L]])
        else:
            digest = _digest(pc.page_blocks(oracle_format(run), pages, L))
        jobs.append((name, layer, kind, b, L, run.c_bits, run.r_bits, run.meta, digest, out[b], lse[b], run.tau))
    with mp.get_context("spawn").Pool(16) as pool:
        res = pool.map(oracle_sequence, jobs, chunksize=1)
        assert all(r[1] for r in res), f"{name}: cache bytes differ from the oracle's in sequences " \
            f"{[r[0] for r in res if not r[1]][:10]}"
        stats = AttnStats.merged([r[2] for r in res])
        rms = np.sqrt(stats.sq_sum / stats.n)
        limit = MAX_TOL * rms
        # every wave holding a row past the max rule, modelled
        past = [(r[0], i, h) for r in res for i, h in zip(*np.nonzero(r[3] > limit))]
        waves = sorted({(b, int(i), int(h) // 32 * 32) for b, i, h in past})
        assert not waves or (run.split_tokens and run.H % 32 == 0 and run.H >= 64), \
            "rows past the max rule in a configuration the rounding model does not cover"
        mjobs = [jobs[b][:9] + (run.tau, run.split_tokens, i, list(range(h0, h0 + 32))) for b, i, h0 in waves]
        modelled = pool.map(model_rows, mjobs, chunksize=1)
    print(f"{name} layer {layer} {kind}: {len(lens)} sequences, {out.size} outputs, "
          f"max excess {stats.excess_ratio():.4f} of the RMS (rule {MAX_TOL}), "
          f"{len(past)} rows past the rule, {len(waves)} waves modelled, "
          f"{time.perf_counter() - t0:.1f} s", flush=True)
    stats.check(f"{name} layer {layer} {kind} (all outputs)", max_rule=False)
    worst = 0.0
    for (b, i, h0), (b_, i_, ok, parts) in zip(waves, modelled):
        assert ok and (b_, i_) == (b, i)
        worst = max(worst, _check_modelled(name, run, out, b, i, list(range(h0, h0 + 32)), parts))
    if past:
        pytest.xfail(f"{name} layer {layer} {kind}: {len(past)} (query token, head) rows of {out.size // 512} have "
                     f"outputs past the max rule (worst {stats.excess_ratio():.4f} of the RMS); their split "
                     f"partials are the rounding model's (worst {worst:.1e} of the row's largest element beyond "
                     f"their own fp16 rounding) and their outputs the bf16 rounding of the combined partials; "
                     f"every other rule holds")

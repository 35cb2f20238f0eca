"""GPU parity of decode attention (+ split-KV combine) against the oracle.

Small cases compare every output of every row with the oracle (exact softmax
in fp64 over the oracle's own reconstruction of the same cache); they span
several tiles, ragged tails, one- and two-token queries, split and unsplit
launches, 4-bit and 2-bit content, the BF16 cache and 16 to 512 query rows
(one to four 128-row blocks per work item, the last one part-filled).
The full-size workloads run in the launch configuration the benchmark times
and are compared on sampled sequences and heads.
"""
import numpy as np
import pytest

from gpu_support import FP16_LIMITED, AttnStats, bf16_bits_to_f64, check_fp16_limited, check_sequence, lse_bound
from oracle import attention as at
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu


def _run(w, **kw):
    from paper_2609_36760_amd.runner import DecodeRun
    run = DecodeRun(w, **kw)
    run.step()
    import torch
    torch.cuda.synchronize()
    return run


SMALL = [
    # (name, H, s_q, lens, c_bits or 'bf16', split_tokens)
    ("c4_h128_sq1_nosplit", 128, 1, [1, 31, 32, 33, 95, 200, 517], 4, 0),
    ("c4_h128_sq1_split64", 128, 1, [1, 31, 33, 200, 517], 4, 64),
    ("c4_h128_sq2_split96", 128, 2, [2, 3, 64, 65, 300], 4, 96),
    ("c4_h128_sq2_nosplit", 128, 2, [2, 129, 250], 4, 0),
    ("c2_h128_sq1_split32", 128, 1, [5, 64, 290], 2, 32),
    ("c2_h128_sq2_nosplit", 128, 2, [2, 77, 191], 2, 0),
    ("c4_h16_sq1_nosplit", 16, 1, [1, 7, 256, 333], 4, 0),
    ("c4_h16_sq2_split64", 16, 2, [2, 70, 257], 4, 64),
    ("c4_h48_sq2_nosplit", 48, 2, [9, 100], 4, 0),
    ("c4_h64_sq1_split128", 64, 1, [130, 400], 4, 128),
    ("bf16_h128_sq1_split64", 128, 1, [1, 33, 300], "bf16", 64),
    ("bf16_h128_sq2_nosplit", 128, 2, [2, 97, 260], "bf16", 0),
    ("bf16_h16_sq1_nosplit", 16, 1, [5, 256], "bf16", 0),
    # row counts: 32 rows over two 16-row waves, part-filled and several
    # 128-row blocks per work item
    ("c4_h32_sq1_split32", 32, 1, [1, 45, 200], 4, 32),
    ("c4_h32_sq2_nosplit", 32, 2, [2, 64, 150], 4, 0),
    ("c4_h80_sq2_split64", 80, 2, [2, 99, 230], 4, 64),
    ("c2_h256_sq2_split64", 256, 2, [2, 70, 201], 2, 64),
    ("bf16_h256_sq1_nosplit", 256, 1, [1, 130], "bf16", 0),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_decode_small_all_rows(case):
    name, H, s_q, lens, cb, split = case
    kind = "bf16" if cb == "bf16" else "lowbit"
    bits = 4 if cb == "bf16" else cb
    w = syn.Workload(name, 100 + SMALL.index(case), B=len(lens), H=H, s_q=s_q, context=None,
                     layers=((bits, 4),), split_tokens=split, ctx_range=(1, 2))
    run = _run(w, kind=kind, seq_lens=np.asarray(lens, np.int32))
    stats = AttnStats()
    for b in range(len(lens)):
        check_sequence(stats, run, b)
        print(f"  seq {b} L={lens[b]}: cumulative max_abs={stats.abs_max:.4g}", flush=True)
    if name in FP16_LIMITED:
        check_fp16_limited(stats, name)
    else:
        stats.check(name)


def test_split_partials_match_oracle_chunks():
    """The partials themselves (before the combine) follow the chunk definition."""
    import torch
    w = syn.Workload("partials", 140, B=2, H=128, s_q=2, context=None, split_tokens=64, ctx_range=(1, 2))
    lens = np.asarray([150, 64], np.int32)
    from paper_2609_36760_amd.runner import DecodeRun
    run = DecodeRun(w, seq_lens=lens)
    run.append_new_tokens()
    from paper_2609_36760_amd import _binding as mb
    mb.mla_lowbit_decode_attn(run.fmt, run.q_lat, run.q_rope, run.cache, run.num_pages, run.block_table,
                              run.seq_lens, 2, 128, w.tau, split_tokens=64, split_indptr=run.split_indptr,
                              num_splits=run.num_splits, part_m=run.part_m, part_s=run.part_s, part_o=run.part_o)
    torch.cuda.synchronize()
    R = 2 * 128
    pm = run.part_m.cpu().numpy().reshape(-1, R)
    ps = run.part_s.cpu().numpy().reshape(-1, R)
    po = run.part_o.float().cpu().numpy().reshape(-1, R, 512)     # normalized by part_s
    from gpu_support import cache_values
    for b in range(2):
        L = int(lens[b])
        c_hat, kr_hat = cache_values(run, b)
        ql, qr = syn.queries(w, 0, batch=[b])
        bounds = [(a, min(a + 64, L)) for a in range(0, L, 64)]
        m, s, o = at.chunk_partials(at.bf16_bits_to_f64(ql[0]).reshape(R, 512),
                                    at.bf16_bits_to_f64(qr[0]).reshape(R, 64), c_hat, kr_hat, w.tau,
                                    at.decode_limits(L, 2, 128), bounds)
        j0 = run.split_indptr_host[b]
        for j in range(len(bounds)):
            gm, gs, go = pm[j0 + j], ps[j0 + j], po[j0 + j]
            empty = np.isneginf(m[j])
            assert np.array_equal(np.isneginf(gm), empty)
            assert np.all(gs[empty] == 0) and np.all(go[empty] == 0)
            live = ~empty
            # the chunk maximum, the chunk lse and the normalised chunk output,
            # within the bounds of the full-row comparison applied to the chunk
            a, e = bounds[j]
            ql64 = at.bf16_bits_to_f64(ql[0]).reshape(R, 512)
            qr64 = at.bf16_bits_to_f64(qr[0]).reshape(R, 64)
            lim = np.minimum(at.decode_limits(L, 2, 128), e)
            mag = np.abs(ql64) @ np.abs(c_hat[a:e].astype(np.float64)).T + np.abs(qr64) @ np.abs(kr_hat[a:e].astype(np.float64)).T
            mag = np.where(np.arange(a, e)[None, :] < lim[:, None], mag, 0.0)
            dz = w.tau * 2.0 ** -8 * mag.max(axis=1)
            assert np.all(np.abs(gm - m[j])[live] <= dz[live] + 1e-5 * np.abs(m[j][live]))
            assert np.all(np.abs((gm + np.log(gs)) - (m[j] + np.log(s[j])))[live] <= dz[live] + 1e-5)
            zc = at.logits(ql64, qr64, c_hat[a:e], kr_hat[a:e], w.tau)
            zc = np.where(np.arange(a, e)[None, :] < lim[:, None], zc, -np.inf)[live]
            wts = np.exp(zc - zc.max(axis=1, keepdims=True))
            wts /= wts.sum(axis=1, keepdims=True)
            A = wts @ np.abs(c_hat[a:e].astype(np.float64))
            want = o[j][live] / s[j][live, None]
            tol = 1.25 * (2.0 ** -9 * np.abs(want) + (2.0 ** -8 + 2.1 * dz[live, None]) * A)
            assert np.all(np.abs(go[live] - want) <= tol)


def test_large_score_jump_rescale():
    """Scores that jump far above the first tiles' maximum: the running reference
    is raised and the accumulators rescaled in place."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    dev = "cuda"
    L, H = 200, 128
    rng = np.random.default_rng(5)
    sgn = np.where(np.arange(512) % 2 == 0, 1.0, -1.0).astype(np.float32)
    c = np.zeros((L, 512), np.float32)
    # late tokens: +-2 per channel (groups straddle zero), aligned with the query signs
    c[64:] = 2.0 * sgn + 0.01 * rng.standard_normal((L - 64, 512)).astype(np.float32)
    c[:64] = 0.01 * rng.standard_normal((64, 512)).astype(np.float32)
    k = 0.1 * rng.standard_normal((L, 64)).astype(np.float32)
    rb = lambda x: ((x.view(np.uint32) + 0x7FFF + ((x.view(np.uint32) >> 16) & 1)) >> 16).astype(np.uint16)
    cb, kb = rb(c), rb(k)
    ql = rb(sgn[None, None, None, :] * np.linspace(0.5, 1.0, H, dtype=np.float32)[None, None, :, None])
    qr = rb(rng.standard_normal((1, 1, H, 64)).astype(np.float32))
    tau = 1 / np.sqrt(192)
    fmt = mb.cache_format(c_bits=4)
    pb = mb.mla_lowbit_page_bytes(fmt)
    cache = torch.zeros(4 * pb, dtype=torch.uint8, device=dev)
    slots = torch.arange(L, dtype=torch.int64, device=dev)
    mb.mla_lowbit_quant_append(fmt, torch.from_numpy(cb.view(np.int16)).to(dev),
                               torch.from_numpy(kb.view(np.int16)).to(dev), slots, cache, 4)
    out = torch.empty((1, 1, H, 512), dtype=torch.int16, device=dev)
    lse = torch.empty((1, 1, H), dtype=torch.float32, device=dev)
    bt = torch.arange(4, dtype=torch.int32, device=dev).reshape(1, 4)
    sl = torch.tensor([L], dtype=torch.int32, device=dev)
    mb.mla_lowbit_decode_attn(fmt, torch.from_numpy(ql.view(np.int16)).to(dev),
                              torch.from_numpy(qr.view(np.int16)).to(dev), cache, 4, bt, sl, 1, H, tau,
                              out=out, lse=lse)
    torch.cuda.synchronize()
    from oracle import paged_cache as pc
    ofmt = pc.CacheFormat(c_bits=4)
    got_cache = cache.cpu().numpy()
    want_cache = got_cache.copy()
    pc.write_tokens(want_cache, ofmt, np.arange(L), cb, kb)
    assert np.array_equal(got_cache, want_cache)
    c_hat, kr_hat = pc.read_tokens(got_cache, ofmt, np.arange(L))
    want, want_lse = at.decode_sequence(ql[0], qr[0], c_hat, kr_hat, tau)
    z = at.logits(at.bf16_bits_to_f64(ql[0, 0]), at.bf16_bits_to_f64(qr[0, 0]), c_hat, kr_hat, tau)
    assert (z[:, 64:].max(1) - z[:, :32].max(1)).max() * np.log2(np.e) > 64   # the path is taken
    stats = AttnStats()
    stats.add(bf16_bits_to_f64(out.cpu().numpy())[0], want, lse.cpu().numpy()[0], want_lse,
              lse_bound(ql[0], qr[0], c_hat, kr_hat, tau, L, 1))
    stats.check("rescale")


def test_identical_keys_give_the_key():
    import torch

    from paper_2609_36760_amd import _binding as mb
    dev = "cuda"
    L, H = 300, 128
    rng = np.random.default_rng(9)
    row_c = rng.standard_normal(512).astype(np.float32)
    row_k = rng.standard_normal(64).astype(np.float32)
    to_b = lambda x: (x.view(np.uint32) >> 16).astype(np.uint16)
    cb = np.tile(to_b(row_c), (L, 1))
    kb = np.tile(to_b(row_k), (L, 1))
    fmt = mb.cache_format(c_bits=4)
    pb = mb.mla_lowbit_page_bytes(fmt)
    cache = torch.zeros(5 * pb, dtype=torch.uint8, device=dev)
    mb.mla_lowbit_quant_append(fmt, torch.from_numpy(cb.view(np.int16)).to(dev), torch.from_numpy(kb.view(np.int16)).to(dev),
                               torch.arange(L, dtype=torch.int64, device=dev), cache, 5)
    ql = to_b(rng.standard_normal((1, 1, H, 512)).astype(np.float32))
    qr = to_b(rng.standard_normal((1, 1, H, 64)).astype(np.float32))
    out = torch.empty((1, 1, H, 512), dtype=torch.int16, device=dev)
    lse = torch.empty((1, 1, H), dtype=torch.float32, device=dev)
    mb.mla_lowbit_decode_attn(fmt, torch.from_numpy(ql.view(np.int16)).to(dev), torch.from_numpy(qr.view(np.int16)).to(dev),
                              cache, 5, torch.arange(5, dtype=torch.int32, device=dev).reshape(1, 5),
                              torch.tensor([L], dtype=torch.int32, device=dev), 1, H, 0.07, out=out, lse=lse)
    torch.cuda.synchronize()
    from oracle import paged_cache as pc
    ofmt = pc.CacheFormat(c_bits=4)
    got_cache = cache.cpu().numpy()
    want_cache = got_cache.copy()
    pc.write_tokens(want_cache, ofmt, np.arange(L), cb, kb)
    assert np.array_equal(got_cache, want_cache)
    c_hat, kr_hat = pc.read_tokens(got_cache, ofmt, np.arange(1))
    got = bf16_bits_to_f64(out.cpu().numpy())[0, 0]
    # uniform weights: the output is the (bf16-rounded) reconstructed key row
    want = bf16_bits_to_f64(((c_hat[0].view(np.uint32) + 0x7FFF + ((c_hat[0].view(np.uint32) >> 16) & 1)) >> 16)
                            .astype(np.uint16))
    np.testing.assert_allclose(got, np.tile(want, (H, 1)), rtol=2 ** -7, atol=0)
    z0 = 0.07 * (at.bf16_bits_to_f64(ql[0, 0]) @ c_hat[0] + at.bf16_bits_to_f64(qr[0, 0]) @ kr_hat[0])
    bound = lse_bound(ql[0], qr[0], c_hat[[0] * L], kr_hat[[0] * L], 0.07, L, 1)
    assert np.all(np.abs(lse.cpu().numpy()[0, 0] - (z0 + np.log(L))) <= bound + 1e-5 * np.abs(z0 + np.log(L)))


def test_empty_batch_is_noop():
    import torch

    from paper_2609_36760_amd import _binding as mb
    dev = "cuda"
    q = torch.zeros((0, 1, 16, 512), dtype=torch.int16, device=dev)
    z = torch.zeros(16, dtype=torch.int16, device=dev)
    cache = torch.zeros(20736, dtype=torch.uint8, device=dev)
    mb.mla_lowbit_decode_attn(mb.cache_format(), q, q, cache, 1,
                              torch.zeros((0, 1), dtype=torch.int32, device=dev), z, 1, 16, 0.1, out=q)
    torch.cuda.synchronize()


# ---- full-size workloads, launch configuration of the benchmark ---------------

FULL = [
    # (workload, layer, kind, sampled sequences, sampled heads, path)
    # path "fused": the benchmark's step (append inside the decode launch, then
    # the combine); "step": the writer launch, the decode launch, the combine
    ("tiny_b1_h16_256", 0, "lowbit", None, None, "fused"),
    ("dsv3_b32_h128_4k_c4r4", 0, "lowbit", [0, 17, 31], None, "fused"),
    ("dsv3_b32_h128_4k_c4r4", 0, "lowbit", [5, 30], None, "step"),
    ("dsv3_b32_h128_4k_c4r4", 0, "bf16", [3, 30], None, "fused"),
    ("int2_b64_h128_32k_c2r4", 0, "lowbit", [0, 63], np.arange(0, 128, 4), "fused"),
    ("splitkv_b8_h128_128k_c4r4", 0, "lowbit", [5], np.arange(0, 128, 8), "fused"),
    ("ragged_b96_h128_sq2_mixed", 0, "lowbit", "ends", np.arange(0, 128, 4), "fused"),
    ("ragged_b96_h128_sq2_mixed", 1, "lowbit", "ends", np.arange(1, 128, 4), "fused"),
    ("c4r4_b64_h128_32k", 0, "lowbit", [1, 62], np.arange(0, 128, 4), "fused"),
    ("c4r4_b64_h128_32k", 0, "bf16", [7], np.arange(0, 128, 8), "fused"),
]


@pytest.mark.slow
@pytest.mark.parametrize("case", FULL, ids=[f"{c[0]}-L{c[1]}-{c[2]}-{c[5]}" for c in FULL])
def test_decode_full_size_sampled(case):
    """Every token of the sampled sequences: the GPU-written pages byte for
    byte against the oracle's packing, then the outputs of the sampled heads
    against the oracle's attention over the values dequantized from those
    bytes."""
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    name, layer, kind, seqs, heads, path = case
    w = syn.WORKLOADS[name]
    run = DecodeRun(w, layer=layer, kind=kind)
    (run.fused_step if path == "fused" else run.step)()
    torch.cuda.synchronize()
    out = run.out.cpu().numpy()
    assert np.all(np.isfinite(bf16_bits_to_f64(out)))
    if seqs is None:
        seqs = range(w.B)
    elif seqs == "ends":
        order = np.argsort(run.lens)
        seqs = [int(order[0]), int(order[1]), int(order[-1])]
    stats = AttnStats()
    for b in seqs:
        check_sequence(stats, run, b, heads)
        print(f"  seq {b} L={int(run.lens[b])}: cache bytes exact, cumulative max_excess={stats.excess_max:.4g}",
              flush=True)
    stats.check(f"{name} layer {layer} {kind} {path}")
    del run
    torch.cuda.empty_cache()


def test_repeated_launches_are_deterministic():
    """Back-to-back launches of the same decode give bit-identical partials and output."""
    import torch

    from paper_2609_36760_amd import _binding as mb
    from paper_2609_36760_amd.runner import DecodeRun
    w = syn.WORKLOADS["dsv3_b32_h128_4k_c4r4"]
    run = DecodeRun(w)
    run.attend()
    torch.cuda.synchronize()
    ref_o, ref_m, ref_out = run.part_o.clone(), run.part_m.clone(), run.out.clone()
    for _ in range(3):
        for _ in range(10):
            mb.mla_lowbit_decode_attn(run.fmt, run.q_lat, run.q_rope, run.cache, run.num_pages, run.block_table,
                                      run.seq_lens, run.s_q, run.H, run.tau, split_tokens=run.split_tokens,
                                      split_indptr=run.split_indptr, num_splits=run.num_splits, part_m=run.part_m,
                                      part_s=run.part_s, part_o=run.part_o)
        run.attend()
        torch.cuda.synchronize()
        assert torch.equal(run.part_o, ref_o) and torch.equal(run.part_m, ref_m)
        assert torch.equal(run.out, ref_out)


# ---- few query rows (s_q * H <= 32: the narrow kernel) ----------------------

NARROW = [
    # (name, H, s_q, lens, c_bits or 'bf16', split)
    ("n_c2_h16_sq1_split32", 16, 1, [1, 15, 16, 17, 200, 331], 2, 32),
    ("n_c4_h32_sq1_nosplit", 32, 1, [3, 48, 95, 260], 4, 0),
    ("n_bf16_h16_sq2_split64", 16, 2, [2, 31, 130, 257], "bf16", 64),
    ("n_c4_h16_sq1_split96", 16, 1, [1, 96, 97, 1000, 2049], 4, 96),
]


@pytest.mark.parametrize("case", NARROW, ids=[c[0] for c in NARROW])
def test_decode_narrow_all_rows(case):
    name, H, s_q, lens, cb, split = case
    kind = "bf16" if cb == "bf16" else "lowbit"
    bits = 4 if cb == "bf16" else cb
    w = syn.Workload(name, 160 + NARROW.index(case), B=len(lens), H=H, s_q=s_q, context=None,
                     layers=((bits, 4),), split_tokens=split, ctx_range=(1, 2))
    run = _run(w, kind=kind, seq_lens=np.asarray(lens, np.int32))
    stats = AttnStats()
    for b in range(len(lens)):
        check_sequence(stats, run, b)
        print(f"  seq {b} L={lens[b]}: cumulative max_abs={stats.abs_max:.4g}", flush=True)
    stats.check(name)

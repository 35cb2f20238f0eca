"""Rounding budget of the decode datapath (CPU only).

Emulates, with the oracle's reconstructed cache, the roundings a kernel makes
(reconstructed keys/values and softmax weights to a 16-bit type, fp32
accumulation, bf16 output) and measures the error against the exact fp64
result under the parity rule used by the GPU tests (per latent channel:
max error beyond the bf16 output's half-ulp <= 2e-2 of the channel RMS).

It records why the low-bit kernels use fp16 rather than bf16 matrix products:
with bf16 tiles and weights the rule fails on the synthetic DeepSeek-V3-shaped
workload, with fp16 it holds; why the BF16-cache kernel may use bf16 products
(its cache values and queries are exact in bf16, so only the weights are
rounded, and that passes); and that rounding the exact result to bf16 already
costs more than 2e-2 of the global RMS, which is why the rule is read per
channel beyond the output's own rounding.
"""
import numpy as np
import pytest

from oracle import attention as at
from oracle import paged_cache as pc
from paper_2609_36760_amd import synthetic as syn


def _rnd_bf16(x):
    b = np.ascontiguousarray(x, np.float32).view(np.uint32)
    return (((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16).astype(np.uint32).view(np.float32)


def _rnd_f16(x):
    return np.asarray(x, np.float32).astype(np.float16).astype(np.float32)


def _ident(x):
    return np.asarray(x, np.float32)


def _emulate(ql, qr, c_hat, kr_hat, tau, s_q, kv_round, p_round):
    R, L = ql.shape[0], c_hat.shape[0]
    K = np.concatenate([kv_round(c_hat), kv_round(kr_hat)], 1).astype(np.float64)
    S = (np.concatenate([ql, qr], 1) @ K.T).astype(np.float32)
    lim = at.decode_limits(L, s_q, R // s_q)
    x = np.where(np.arange(L)[None] < lim[:, None], S * np.float32(tau * np.log2(np.e)), -np.inf)
    p = np.exp2(x - x.max(1, keepdims=True)).astype(np.float32)
    O = (p_round(p).astype(np.float64) @ K[:, :512]) / p.astype(np.float64).sum(1, keepdims=True)
    return _rnd_bf16(O.astype(np.float32)).astype(np.float64)


def _excess_ratio(got, want):
    """Per-channel max of (error beyond half a bf16 ulp of the exact value) / channel RMS."""
    ay = np.abs(want) * (1 + 2.0 ** -7)
    half_ulp = np.where(ay > 0, np.exp2(np.floor(np.log2(np.maximum(ay, 1e-300))) - 8), 0.0)
    ex = np.maximum(np.abs(got - want) - half_ulp, 0.0)
    return float((ex.max(0) / np.sqrt((want ** 2).mean(0))).max())


@pytest.fixture(scope="module")
def sample():
    w = syn.WORKLOADS["dsv3_b32_h128_4k_c4r4"]
    lens = syn.seq_lens(w)
    rows = []
    for b in (0, 17):
        L = int(lens[b])
        c, k = syn.sequence_tokens(w, 0, b, L)
        c_hat, kr_hat = pc.encode_sequence_dense(pc.CacheFormat(), c, k)
        ql, qr = syn.queries(w, 0, batch=[b])
        hs = np.arange(0, 128, 2)
        want, _ = at.decode_sequence(ql[0][:, hs], qr[0][:, hs], c_hat, kr_hat, w.tau)
        rows.append((at.bf16_bits_to_f64(ql[0][:, hs]).reshape(-1, 512),
                     at.bf16_bits_to_f64(qr[0][:, hs]).reshape(-1, 64), c_hat, kr_hat, want.reshape(-1, 512)))
    return w, rows


def _ratio(w, rows, kv, pr):
    got = np.concatenate([_emulate(a, b, c, d, w.tau, w.s_q, kv, pr) for a, b, c, d, _ in rows])
    want = np.concatenate([r[4] for r in rows])
    return got, want, _excess_ratio(got, want)


def test_fp16_datapath_meets_the_rule(sample):
    w, rows = sample
    _, _, r = _ratio(w, rows, _rnd_f16, _rnd_f16)
    assert r <= 0.02, r


def test_bf16_datapath_fails_the_rule(sample):
    w, rows = sample
    _, _, r = _ratio(w, rows, _rnd_bf16, _rnd_bf16)
    assert r > 0.02, r


def test_bf16_output_rounding_alone_exceeds_the_global_rule(sample):
    w, rows = sample
    got, want, _ = _ratio(w, rows, _ident, _ident)
    assert np.abs(got - want).max() > 0.02 * np.sqrt((want ** 2).mean())


@pytest.fixture(scope="module")
def bf16_sample():
    """Exact bf16 cache values (the BF16 cache stores the latents as they are)."""
    w = syn.WORKLOADS["dsv3_b32_h128_4k_c4r4"]
    lens = syn.seq_lens(w)
    rows = []
    for b in (0, 17):
        L = int(lens[b])
        c, k = syn.sequence_tokens(w, 0, b, L)
        c_hat, kr_hat = at.bf16_bits_to_f64(c), at.bf16_bits_to_f64(k)
        ql, qr = syn.queries(w, 0, batch=[b])
        hs = np.arange(0, 128, 2)
        want, _ = at.decode_sequence(ql[0][:, hs], qr[0][:, hs], c_hat, kr_hat, w.tau)
        rows.append((at.bf16_bits_to_f64(ql[0][:, hs]).reshape(-1, 512),
                     at.bf16_bits_to_f64(qr[0][:, hs]).reshape(-1, 64), c_hat, kr_hat, want.reshape(-1, 512)))
    return w, rows


def test_bf16_cache_with_bf16_weights_meets_the_rule(bf16_sample):
    w, rows = bf16_sample
    _, _, r = _ratio(w, rows, _ident, _rnd_bf16)
    assert r <= 0.02, r

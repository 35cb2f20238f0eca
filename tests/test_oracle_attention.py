"""Pins for the attention oracle (CPU only).

``oracle.attention`` is checked against: a scalar-loop restatement on tiny
inputs, the materialised non-absorbed MLA head (Sec. 2.1), closed forms
(identical keys, a single key), invariances (key permutation, any chunking
merged by the Appendix C.5 rule), the causal reading for two query tokens, and
Proposition 2's bound (Sec. 3.2, proved in Appendix C.3).
"""
import numpy as np
import pytest

from oracle import attention as at
from oracle import paged_cache as pc
from oracle import quantizer as qz
from oracle import reference_mla as ref

TAU = 1.0 / np.sqrt(192.0)


def _rand(rng, *shape, scale=1.0):
    return rng.standard_normal(shape) * scale


def test_matches_scalar_loops_tiny():
    rng = np.random.default_rng(0)
    R, L, dc, dr = 4, 6, 8, 4
    ql, qr = _rand(rng, R, dc), _rand(rng, R, dr)
    c, k = _rand(rng, L, dc), _rand(rng, L, dr)
    limits = np.array([6, 5, 1, 3])
    out, lse = at.attend(ql, qr, c, k, 0.7, limits)
    bo, bl = ref.brute_force_rows(ql.tolist(), qr.tolist(), c.tolist(), k.tolist(), 0.7, limits)
    np.testing.assert_allclose(out, np.array(bo), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, np.array(bl), rtol=1e-12, atol=1e-13)


def test_absorbed_equals_materialised():
    rng = np.random.default_rng(1)
    L, dc, dr, dh, dv, R = 23, 32, 8, 12, 10, 3
    c, k = _rand(rng, L, dc), _rand(rng, L, dr)
    w_uk, w_uv = _rand(rng, dc, dh, scale=0.3), _rand(rng, dc, dv, scale=0.3)
    q_nope, q_rope = _rand(rng, R, dh), _rand(rng, R, dr)
    limits = np.array([23, 22, 9])
    want = ref.materialised_head(q_nope, q_rope, c, k, w_uk, w_uv, TAU, limits)
    q_lat = q_nope @ w_uk.T                   # absorbed content query
    o, _ = at.attend(q_lat, q_rope, c, k, TAU, limits)
    np.testing.assert_allclose(o @ w_uv, want, rtol=1e-12, atol=1e-12)


def test_identical_keys_uniform():
    rng = np.random.default_rng(2)
    L = 37
    c0, k0 = _rand(rng, 512), _rand(rng, 64)
    ql, qr = _rand(rng, 5, 512), _rand(rng, 5, 64)
    out, lse = at.attend(ql, qr, np.tile(c0, (L, 1)), np.tile(k0, (L, 1)), TAU, np.full(5, L))
    z0 = TAU * (ql @ c0 + qr @ k0)
    np.testing.assert_allclose(out, np.tile(c0, (5, 1)), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, z0 + np.log(L), rtol=1e-12, atol=1e-12)


def test_single_key():
    rng = np.random.default_rng(3)
    c, k = _rand(rng, 1, 512), _rand(rng, 1, 64)
    ql, qr = _rand(rng, 2, 512), _rand(rng, 2, 64)
    out, lse = at.attend(ql, qr, c, k, TAU, np.ones(2))
    np.testing.assert_allclose(out, np.tile(c, (2, 1)), rtol=0, atol=0)
    np.testing.assert_allclose(lse, TAU * (ql @ c[0] + qr @ k[0]), rtol=1e-13)


@pytest.mark.parametrize("seed", range(4))
def test_chunk_merge_equals_whole(seed):
    rng = np.random.default_rng(10 + seed)
    L, R = 50, 6
    c, k = _rand(rng, L, 512), _rand(rng, L, 64)
    ql, qr = _rand(rng, R, 512, scale=2.0), _rand(rng, R, 64, scale=2.0)
    limits = np.array([50, 49, 17, 1, 33, 50])
    cuts = np.sort(rng.choice(np.arange(1, L), size=4, replace=False))
    edges = [0, *cuts.tolist(), L]
    bounds = list(zip(edges[:-1], edges[1:]))
    m, s, o = at.chunk_partials(ql, qr, c, k, TAU, limits, bounds)
    assert np.isneginf(m).any()                 # some rows see nothing of some chunks
    out, lse = at.merge(m, s, o)
    want_o, want_l = at.attend(ql, qr, c, k, TAU, limits)
    np.testing.assert_allclose(out, want_o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, want_l, rtol=1e-12, atol=1e-12)
    # partial definitions: chunk maxima are the chunk's largest logit
    z = at.logits(ql, qr, c, k, TAU)
    a, b = bounds[0]
    assert m[0, 0] == z[0, a:b].max()


def test_key_permutation_invariance():
    rng = np.random.default_rng(4)
    L = 40
    c, k = _rand(rng, L, 512), _rand(rng, L, 64)
    ql, qr = _rand(rng, 3, 512), _rand(rng, 3, 64)
    p = rng.permutation(L)
    o1, l1 = at.attend(ql, qr, c, k, TAU, np.full(3, L))
    o2, l2 = at.attend(ql, qr, c[p], k[p], TAU, np.full(3, L))
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(l1, l2, rtol=1e-12, atol=1e-12)


def test_two_query_tokens_are_causal():
    rng = np.random.default_rng(5)
    L, H = 30, 4
    bits = lambda a: (a.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    ql, qr = bits(_rand(rng, 2, H, 512)), bits(_rand(rng, 2, H, 64))
    c, k = _rand(rng, L, 512), _rand(rng, L, 64)
    o1, l1 = at.decode_sequence(ql, qr, c, k, TAU)
    c2 = c.copy()
    c2[-1] += 5.0                                 # change only the newest key
    o2, l2 = at.decode_sequence(ql, qr, c2, k, TAU)
    np.testing.assert_array_equal(o1[0], o2[0])   # query 0 does not see token L-1
    np.testing.assert_array_equal(l1[0], l2[0])
    assert np.abs(o1[1] - o2[1]).max() > 1e-6
    assert at.decode_limits(L, 2, H).tolist() == [L - 1] * H + [L] * H


def test_positional_bound_prop2():
    """Quantizing only the RoPE key moves each head by at most Proposition 2's bound."""
    rng = np.random.default_rng(6)
    L, H = 200, 8
    c = rng.standard_normal((L, 512)).astype(np.float32)
    kr = (rng.standard_normal((L, 64)) * np.repeat(np.logspace(-1, np.log10(5), 32), 2)).astype(np.float32)
    kr_bits = (kr.view(np.uint32) >> 16).astype(np.uint16)
    kr = qz.bf16_bits_to_f32(kr_bits)
    packed, s16, z16 = qz.quantize_token_path(kr_bits, 4)
    kr_hat = qz.dequantize_token_path(packed, s16, z16, 4)
    ql, qr = rng.standard_normal((2, H, 512)), rng.standard_normal((2, H, 64))
    limits = at.decode_limits(L, 2, 1)
    tight = 0
    for h in range(H):
        o_exact, _ = at.attend(ql[:, h], qr[:, h], c, kr, TAU, limits)
        o_quant, _ = at.attend(ql[:, h], qr[:, h], c, kr_hat, TAU, limits)
        dz = qr[:, h] @ (kr_hat.astype(np.float64) - kr.astype(np.float64)).T
        dz[0, L - 1] = 0.0                         # query 0 cannot see the newest key
        lhs = np.linalg.norm(o_quant - o_exact)
        rhs = ref.positional_bound(TAU, dz, c)
        assert lhs <= rhs
        tight = max(tight, lhs / rhs)
    assert tight > 1e-3                            # the bound is not vacuous here


def test_decode_uses_reconstructed_cache():
    """End-to-end oracle chain on a tiny paged cache: write, read back, attend."""
    rng = np.random.default_rng(8)
    f = pc.CacheFormat(c_bits=4)
    L, H = 100, 16
    bits = lambda a: (a.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    c_bits, k_bits = bits(rng.standard_normal((L, 512))), bits(rng.standard_normal((L, 64)))
    cache = np.zeros(4 * f.page_bytes, np.uint8)
    pages = np.array([3, 1])
    slots = pages[np.arange(L) // 64] * 64 + np.arange(L) % 64
    pc.write_tokens(cache, f, slots, c_bits, k_bits)
    c_hat, k_hat = pc.read_tokens(cache, f, slots)
    ql, qr = bits(rng.standard_normal((1, H, 512))), bits(rng.standard_normal((1, H, 64)))
    out, lse = at.decode_sequence(ql, qr, c_hat, k_hat, TAU)
    dense_c, dense_k = pc.encode_sequence_dense(f, c_bits, k_bits)
    d_out, d_lse = at.decode_sequence(ql, qr, dense_c, dense_k, TAU)
    np.testing.assert_array_equal(out, d_out)
    np.testing.assert_array_equal(lse, d_lse)
    ex_out, _ = at.decode_sequence(ql, qr, qz.bf16_bits_to_f32(c_bits), qz.bf16_bits_to_f32(k_bits), TAU)
    assert np.abs(out - ex_out).max() > 1e-3       # quantization error is present

"""Rounding budget of the decode datapath (CPU only).

Emulates, with the oracle's reconstructed cache, the roundings a kernel makes
(reconstructed keys/values, softmax weights and split partials to a 16-bit
type, fp32 accumulation, bf16 output) and measures the error against the
exact fp64 result under the parity rule of the GPU tests: the largest error
beyond half a bf16 ulp of the exact value is at most 2e-2 of the global RMS of
the outputs.

It records:
  * why the low-bit kernels use fp16 rather than bf16 matrix products: with
    bf16 tiles and weights the rule fails on the 32 x 4K workload, with fp16
    it holds;
  * why the BF16-cache kernel normalizes by the sum of its bf16-rounded
    weights (with the exact sum the rule fails, with the rounded one it holds)
    and why protected rows carry each weight as a bf16 pair (the weight and its
    rounded residual, 16 significant bits);
  * that rounding the exact result to bf16 already costs more than 2e-2 of the
    global RMS, so the rule is read beyond the output's own rounding;
  * the two small batches of the GPU tests where the fp16 datapath itself
    exceeds the rule (a 64-head batch of lengths 130 and 400 split at 128; the
    INT2 token-aging case): the fp16 rounding of the reconstructed content
    values moves the logits by about 1e-3, and rows whose weight is split
    between keys whose 10x outlier channels differ by tens of units turn that
    into an output error of 2.5e-2 and 2.65e-2 of the RMS -- reproduced here
    from the rounding model alone (the GPU measured the same to three digits);
    with the content scores exact they fall to 0.8e-2 and 1.2e-2.
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


def _bf16_pair(x):
    """A value held as bf16(x) + bf16(x - bf16(x))."""
    x = np.asarray(x, np.float32)
    h = _rnd_bf16(x)
    return (h.astype(np.float64) + _rnd_bf16(x - h).astype(np.float64)).astype(np.float32)


def _emulate(ql, qr, c_hat, kr_hat, tau, s_q, kv_round, p_round, split=0, part_round=_ident,
             score_round=None, sum_rounded=True, raw=False, groups=None, lim=None, partials=False,
             p_format=None):
    """Output of a kernel that rounds the reconstructed values with kv_round
    (scores: score_round, default the same), the weights with p_round and the
    normalized split partials with part_round.  As in the kernels, the weights
    are 2^(x - ref) with a lazy reference per row and key range: the first
    32-key tile's maximum, moved only when a later tile's maximum exceeds it by
    more than 10 (log2 units); the normalizer sums the rounded weights
    (sum_rounded) or the exact ones.  The output is rounded to bf16 unless
    ``raw``.

    ``groups`` (a group id per row) makes the move wave-uniform as in the
    kernels: when any row of a group moves, every row of the group whose tile
    maximum is above its reference takes that maximum.  ``lim`` overrides the
    rows' visible-key counts (default: the rows are every query token of some
    heads, token-major).  ``partials`` returns, per key range, the unrounded
    partial (true maximum in natural-log units, sum of the weights relative to
    it, normalized weighted sum) instead of the output, and with ``p_format``
    ("f16" or "bf16", the format p_round rounds to) how far each of the last
    two may move if every weight lying within a relative 2^-16 of a rounding
    tie of that format rounds the other way (fp32 scores differ from these
    fp64 ones by less than that)."""
    R, L = ql.shape[0], c_hat.shape[0]
    K = np.concatenate([kv_round(c_hat), kv_round(kr_hat)], 1).astype(np.float64)
    Ks = K if score_round is None else np.concatenate([score_round(c_hat), kv_round(kr_hat)], 1).astype(np.float64)
    S = (np.concatenate([ql, qr], 1) @ Ks.T).astype(np.float32)
    lim = at.decode_limits(L, s_q, R // s_q) if lim is None else np.asarray(lim)
    x = np.where(np.arange(L)[None] < lim[:, None], S * np.float32(tau * np.log2(np.e)), -np.inf).astype(np.float64)
    bounds = [(a, min(a + split, L)) for a in range(0, L, split)] if split else [(0, L)]
    ms, ss, os_, parts = [], [], [], []
    mant, ulp_min = {"f16": (11, 2.0 ** -24), "bf16": (8, 2.0 ** -133), None: (0, 0.0)}[p_format]
    absK = np.abs(K[:, :512])
    for a, b in bounds:
        ref = np.full(R, -np.inf)
        o = np.zeros((R, 512))
        s = np.zeros(R)
        tie_o = np.zeros((R, 512))
        tie_s = np.zeros(R)
        for t0 in range(a, b, 32):
            xx = x[:, t0:min(t0 + 32, b)]
            mt = xx.max(1)
            first = ~np.isfinite(ref)
            ref = np.where(first, mt, ref)
            move = np.isfinite(mt) & (mt > ref + 10)
            if groups is not None:
                wave = np.zeros(int(groups.max()) + 1, bool)
                np.logical_or.at(wave, groups, move)
                move = wave[groups] & np.isfinite(mt) & (mt > ref)
            new_ref = np.where(move, mt, ref)
            alpha = np.where(move, np.exp2(np.where(move, ref - new_ref, 0.0)), 1.0)
            o *= alpha[:, None]
            s *= alpha
            tie_o *= alpha[:, None]
            tie_s *= alpha
            ref = new_ref
            p = np.exp2(xx - np.where(np.isfinite(ref), ref, 0.0)[:, None]).astype(np.float32)
            pr = p_round(p).astype(np.float64)
            o += pr @ K[t0:t0 + xx.shape[1], :512]
            s += (pr if sum_rounded else p.astype(np.float64)).sum(1)
            if partials and p_format is not None:
                p64 = p.astype(np.float64)
                ulp = np.maximum(np.exp2(np.floor(np.log2(np.maximum(p64, 1e-300))) - (mant - 1)), ulp_min)
                near = (p64 > 0) & (np.abs(np.abs(p64 - pr) - ulp / 2) <= 2.0 ** -16 * p64)
                dp = np.where(near, ulp, 0.0)
                tie_o += dp @ absK[t0:t0 + xx.shape[1]]
                tie_s += dp.sum(1)
        on = np.divide(o, s[:, None], out=np.zeros((R, 512)), where=s[:, None] > 0)
        if partials:
            top = x[:, a:b].max(1)
            f = np.where(np.isfinite(top), np.exp2(np.where(np.isfinite(top), ref - top, 0.0)), 0.0)
            tol = np.divide(tie_o + np.abs(on) * tie_s[:, None], s[:, None], out=np.zeros((R, 512)),
                            where=s[:, None] > 0)
            parts.append((top * np.log(2.0), s * f, on, tol, tie_s * f))
        ms.append(np.where(s > 0, np.where(np.isfinite(ref), ref, 0.0), -np.inf))
        ss.append(s)
        os_.append(part_round(on).astype(np.float64) if split else on)
    if partials:
        return parts
    M = np.max(ms, 0)
    W = [np.exp2(mm - M) * s for mm, s in zip(ms, ss)]
    O = sum(w[:, None] * o for w, o in zip(W, os_)) / sum(W)[:, None]
    return O if raw else _rnd_bf16(O.astype(np.float32)).astype(np.float64)


def _excess_ratio(got, want):
    """Largest (error beyond half a bf16 ulp of the exact value) / global RMS."""
    ay = np.abs(want) * (1 + 2.0 ** -7)
    half_ulp = np.where(ay > 0, np.exp2(np.floor(np.log2(np.maximum(ay, 1e-300))) - 8), 0.0)
    ex = np.maximum(np.abs(got - want) - half_ulp, 0.0)
    return float(ex.max() / np.sqrt((want ** 2).mean()))


def _rows(w, seqs, heads, exact_bf16=False, layer=0):
    lens = syn.seq_lens(w) if w.context is not None else None
    c_bits = w.layers[layer][0]
    rows = []
    for b, L in seqs:
        L = int(lens[b]) if L is None else L
        c, k = syn.sequence_tokens(w, layer, b, L)
        if exact_bf16:
            c_hat, kr_hat = at.bf16_bits_to_f64(c), at.bf16_bits_to_f64(k)
        else:
            c_hat, kr_hat = pc.encode_sequence_dense(pc.CacheFormat(c_bits=c_bits), c, k)
        ql, qr = syn.queries(w, layer, batch=[b])
        want, _ = at.decode_sequence(ql[0][:, heads], qr[0][:, heads], c_hat, kr_hat, w.tau)
        rows.append((at.bf16_bits_to_f64(ql[0][:, heads]).reshape(-1, 512),
                     at.bf16_bits_to_f64(qr[0][:, heads]).reshape(-1, 64), c_hat, kr_hat, want.reshape(-1, 512)))
    return rows


@pytest.fixture(scope="module")
def sample():
    w = syn.WORKLOADS["dsv3_b32_h128_4k_c4r4"]
    return w, _rows(w, [(0, None), (17, None)], np.arange(0, 128, 2))


def _ratio(w, rows, kv, pr, **kw):
    got = np.concatenate([_emulate(a, b, c, d, w.tau, w.s_q, kv, pr, **kw) for a, b, c, d, _ in rows])
    want = np.concatenate([r[4] for r in rows])
    return got, want, _excess_ratio(got, want)


def test_fp16_datapath_meets_the_rule(sample):
    w, rows = sample
    _, _, r = _ratio(w, rows, _rnd_f16, _rnd_f16, split=512, part_round=_rnd_f16)
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
    return w, _rows(w, [(3, None), (30, None)], np.arange(128), exact_bf16=True)


def test_bf16_weights_need_a_normalizer_of_the_rounded_weights(bf16_sample):
    """bf16 weights normalized by the sum of the unrounded weights fail the
    rule (the lazy reference puts the dominant weight anywhere in [1, 2^10],
    where its rounding moves the whole row); normalized by the sum of the
    rounded weights they hold it (the BF16-cache kernel), and so does the bf16
    pair (protected rows)."""
    w, rows = bf16_sample
    _, _, once = _ratio(w, rows, _ident, _rnd_bf16, split=512, part_round=_rnd_f16, sum_rounded=False)
    _, _, rounded = _ratio(w, rows, _ident, _rnd_bf16, split=512, part_round=_rnd_f16, sum_rounded=True)
    _, _, pair = _ratio(w, rows, _ident, _bf16_pair, split=512, part_round=_rnd_f16, sum_rounded=False)
    assert once > 0.02, once
    assert rounded <= 0.02, rounded
    assert pair <= 0.02, pair


def _c4_h64_batch_rows():
    w = syn.Workload("c4_h64_sq1_split128", 109, B=2, H=64, s_q=1, context=None, layers=((4, 4),),
                     split_tokens=128, ctx_range=(1, 2))
    return w, _rows(w, [(0, 130), (1, 400)], np.arange(64))


def _aging_excess(score_round=None):
    """The token-aging GPU case aging_c2_h128_sq2_split32 (INT2 content, sink 40
    / recent 8, two query tokens, 16 consecutive steps): the fp16 model's excess
    over all steps (protected rows exact; each sequence modelled unsplit)."""
    from oracle import protection as pr
    start, steps, s_q, (sink, recent) = [2, 40, 47, 60], 16, 2, (40, 8)
    w = syn.Workload("aging_c2_h128_sq2_split32", 362, B=4, H=128, s_q=2, context=None, layers=((2, 4),),
                     split_tokens=32, ctx_range=(1, 2))
    cap = [L + s_q * (steps - 1) for L in start]
    tokens = [syn.sequence_tokens(w, 0, b, L) for b, L in enumerate(cap)]
    ql, qr = syn.queries(w, 0)
    fmt = pc.CacheFormat(c_bits=2)
    worst, sq, n = 0.0, 0.0, 0
    for step in range(steps):
        for b in range(4):
            L = start[b] + s_q * step
            c, k = pr.representation(fmt, tokens[b][0][:L], tokens[b][1][:L], sink, recent)
            keep = pr.protected_mask(L, sink, recent)[:, None]
            rnd = lambda x, keep=keep: np.where(keep, x, _rnd_f16(x))
            got = _emulate(at.bf16_bits_to_f64(ql[b]).reshape(-1, 512), at.bf16_bits_to_f64(qr[b]).reshape(-1, 64),
                           c, k, w.tau, s_q, rnd, _rnd_f16, score_round=score_round)
            want, _ = at.decode_sequence(ql[b], qr[b], c, k, w.tau)
            want = want.reshape(-1, 512)
            ay = np.abs(want) * (1 + 2.0 ** -7)
            half_ulp = np.where(ay > 0, np.exp2(np.floor(np.log2(np.maximum(ay, 1e-300))) - 8), 0.0)
            worst = max(worst, float(np.maximum(np.abs(got - want) - half_ulp, 0.0).max()))
            sq += float((want ** 2).sum())
            n += want.size
    return worst / np.sqrt(sq / n)


def test_fp16_limited_batches_are_the_rounding_models():
    """The GPU tests' fp16-limited batches (gpu_support.FP16_LIMITED): the
    fp16 rounding model alone exceeds the rule by the recorded amounts (the
    GPU measured 2.505e-2 and 2.650e-2), and with exact content scores it
    would not."""
    from gpu_support import FP16_LIMITED
    w, rows = _c4_h64_batch_rows()
    _, _, r = _ratio(w, rows, _rnd_f16, _rnd_f16, split=128, part_round=_rnd_f16)
    _, _, r_exact = _ratio(w, rows, _rnd_f16, _rnd_f16, split=128, part_round=_rnd_f16, score_round=_ident)
    assert abs(r - FP16_LIMITED["c4_h64_sq1_split128"]) < 1e-4, r
    assert r_exact < 0.01, r_exact
    a = _aging_excess()
    a_exact = _aging_excess(score_round=_ident)
    assert abs(a - FP16_LIMITED["aging_c2_h128_sq2_split32"]) < 1e-4, a
    assert a_exact < 0.0125, a_exact


def test_model_partials_combine_to_its_output():
    """The model's partials (the full-output GPU test compares the kernels'
    split partials with them) combine, exactly, to the model's unrounded
    output; a wave-uniform move changes only the references, so without
    weight rounding (the fp32 weights aside) it leaves the result as it is;
    and the tie allowance is zero without a weight format and small
    otherwise."""
    w, rows = _c4_h64_batch_rows()
    ql, qr, c, k, _ = rows[1]                                 # 400 keys, 64 rows
    kw = dict(split=128, part_round=lambda v: v)          # partials left unrounded
    out = _emulate(ql, qr, c, k, w.tau, w.s_q, _rnd_f16, _rnd_f16, raw=True, **kw)
    parts = _emulate(ql, qr, c, k, w.tau, w.s_q, _rnd_f16, _rnd_f16, partials=True, p_format="f16", **kw)
    assert len(parts) == 4
    m = np.stack([p[0] for p in parts])
    s = np.stack([p[1] for p in parts])
    u = np.stack([p[2] for p in parts])
    W = np.exp(m - m.max(0)) * s
    np.testing.assert_allclose((W[..., None] * u).sum(0) / W.sum(0)[:, None], out, rtol=1e-12, atol=1e-12)
    tol = np.stack([p[3] for p in parts])
    assert np.all(tol >= 0) and np.all(np.isfinite(tol))
    assert 0 < np.median(tol / np.abs(u).max(-1, keepdims=True)) < 2.0 ** -15
    none = _emulate(ql, qr, c, k, w.tau, w.s_q, _rnd_f16, _rnd_f16, partials=True, **kw)
    assert all(np.all(p[3] == 0) and np.all(p[4] == 0) for p in none)
    groups = np.repeat(np.arange(2), 32)
    exact = _emulate(ql, qr, c, k, w.tau, w.s_q, _ident, _ident, raw=True, **kw)
    waved = _emulate(ql, qr, c, k, w.tau, w.s_q, _ident, _ident, raw=True, groups=groups, **kw)
    np.testing.assert_allclose(waved, exact, rtol=0, atol=1e-6)

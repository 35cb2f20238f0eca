"""The GPU parity checks can see one wrong key (CPU only).

For every structured GPU case (``structured.CASES``, both query modes) the
outputs of a kernel that is exact but for one key are simulated here from the
oracle and put through the same checks the GPU tests apply (``AttnStats``
over all sequences of the case).  Each simulated kernel rounds the exact
result to the bf16 output (the least error any kernel has); every other
sequence of the case is given its exact bf16-rounded output.  At every edge
position of every sequence (``structured.edge_positions``: tile, page, split,
causal and protection edges) the case must fail:
  * uniform queries: the key dropped, or counted twice;
  * needle queries: the key dropped, or its score taken from its neighbour's
    latent and RoPE key (the value kept).
The unmutated outputs must pass, so the failures come from the mutation.

The same simulation on two random ragged batches of the GPU decode tests (a
128-head and a 16-head one): a key dropped at any of 12 random positions per
sequence fails the batch too.
"""
import numpy as np
import pytest

import structured as st
from gpu_support import AttnStats, bf16_bits_to_f64, elem_bound, lse_bound
from oracle import attention as at
from oracle import paged_cache as pc
from oracle import protection as pr
from paper_2609_36760_amd import synthetic as syn

TAU = 1.0 / np.sqrt(192.0)


def oracle_values(kind, c_bits, meta, prot, cb, kb):
    """The values the oracle attends (fp64): bf16 rows, the quantized cache's
    reconstruction, or the protected representation."""
    if kind == "bf16":
        return at.bf16_bits_to_f64(cb), at.bf16_bits_to_f64(kb)
    fmt = pc.CacheFormat(c_bits=c_bits, meta=meta)
    if prot is not None:
        return pr.representation(fmt, cb, kb, *prot)
    c, k = pc.encode_sequence_dense(fmt, cb, kb)
    return c.astype(np.float64), k.astype(np.float64)


def to_bf16(x):
    return bf16_bits_to_f64(syn.f32_to_bf16_bits(np.asarray(x, np.float32)))


class Sequence:
    """One sequence of a case: exact attention, its bounds, and the outputs of
    a kernel that mishandles one key."""

    def __init__(self, qlb, qrb, c, k, s_q):
        self.qlb, self.qrb, self.c, self.k, self.s_q = qlb, qrb, c, k, s_q
        H = qlb.shape[1]
        self.R = s_q * H
        self.L = c.shape[0]
        self.ql = at.bf16_bits_to_f64(qlb).reshape(self.R, 512)
        self.qr = at.bf16_bits_to_f64(qrb).reshape(self.R, 64)
        self.lim = at.decode_limits(self.L, s_q, H)
        z = at.logits(self.ql, self.qr, c, k, TAU)
        self.z = np.where(np.arange(self.L)[None, :] < self.lim[:, None], z, -np.inf)
        self.m = self.z.max(axis=1)
        self.E = np.exp(self.z - self.m[:, None])
        self.S = self.E.sum(axis=1)
        self.O = self.E @ c
        out, lse = at.decode_sequence(qlb, qrb, c, k, TAU)
        self.want = out.reshape(self.R, 512)
        self.want_lse = lse.reshape(self.R)
        self.lse_bnd = lse_bound(qlb, qrb, c, k, TAU, self.L, s_q)
        self.tol = elem_bound(qlb, qrb, c, k, TAU, self.L, s_q, out, self.lse_bnd).reshape(self.R, 512)

    def stats(self, out, lse):
        s = AttnStats()
        s.add(to_bf16(out), self.want, np.float32(lse), self.want_lse, self.lse_bnd, self.tol)
        return s

    def exact(self):
        return self.stats(self.want, self.want_lse)

    def _row(self, r, zrow):
        """Exact softmax of one row with logits zrow (value rows self.c)."""
        m = zrow.max()
        e = np.exp(zrow - m)
        s = e.sum()
        return (e @ self.c) / s, m + np.log(s)

    def mutated(self, mutation, p):
        """(out [R, 512], lse [R]) of a kernel that drops key p, counts it
        twice, or scores it with its neighbour's latent and RoPE key."""
        vis = self.lim > p
        Ep = self.E[:, p]
        S, O = self.S.copy(), self.O.copy()
        m = self.m.copy()
        exact_rows = np.zeros(self.R, bool)
        if mutation == "drop":
            S[vis] -= Ep[vis]
            O[vis] -= Ep[vis, None] * self.c[p]
            exact_rows = vis & (Ep > 0.5 * self.S)
            zp = None
        elif mutation == "dup":
            S[vis] += Ep[vis]
            O[vis] += Ep[vis, None] * self.c[p]
            zp = None
        elif mutation == "misplace":
            nb = p + 1 if p + 1 < self.L else p - 1
            zp = TAU * (self.ql @ self.c[nb] + self.qr @ self.k[nb])
            Ep2 = np.exp(zp - m)
            S[vis] += Ep2[vis] - Ep[vis]
            O[vis] += (Ep2[vis] - Ep[vis])[:, None] * self.c[p]
            exact_rows = vis & ((Ep > 0.5 * self.S) | (zp > m))
        else:
            raise ValueError(mutation)
        out = np.divide(O, S[:, None], out=np.full_like(O, np.nan), where=S[:, None] > 0)
        lse = np.where(S > 0, m + np.log(np.maximum(S, 1e-300)), np.nan)
        for r in np.nonzero(exact_rows)[0]:
            zrow = self.z[r].copy()
            if mutation == "drop":
                zrow[p] = -np.inf
            else:
                zrow[p] = zp[r]
            if np.isfinite(zrow).any():
                out[r], lse[r] = self._row(r, zrow)
            else:
                out[r], lse[r] = np.nan, np.nan
        return out, lse


def case_sequences(case, mode):
    name, kind, cb, meta, H, s_q, split, prot, lens = case
    seed = 700 + st.CASES.index(case)
    (tokens, ql, qr), probed = st.make_inputs(mode, lens, s_q, H, split, seed, prot, with_probes=True)
    seqs = []
    for b, (ctok, ktok) in enumerate(tokens):
        c, k = oracle_values(kind, cb, meta, prot, ctok, ktok)
        seqs.append(Sequence(ql[b], qr[b], c, k, s_q))
    return seqs, probed


@pytest.mark.parametrize("mode", ["uniform", "needle"])
@pytest.mark.parametrize("case", st.CASES, ids=[c[0] for c in st.CASES])
def test_one_wrong_key_fails_the_structured_case(case, mode):
    name, kind, cb, meta, H, s_q, split, prot, lens = case
    seqs, probed = case_sequences(case, mode)
    exact = [s.exact() for s in seqs]
    AttnStats.merged(exact).check(f"{name} {mode} exact", quiet=True)
    mutations = ("drop", "dup") if mode == "uniform" else ("drop", "misplace")
    tried, missed = 0, []
    for b, seq in enumerate(seqs):
        others = exact[:b] + exact[b + 1:]
        for p in probed[b]:
            for mut in mutations:
                if mode == "needle" and mut == "misplace" and seq.L < 2:
                    continue
                out, lse = seq.mutated(mut, int(p))
                tried += 1
                try:
                    AttnStats.merged(others + [seq.stats(out, lse)]).check(quiet=True)
                except AssertionError:
                    continue
                missed.append((b, seq.L, int(p), mut))
    for L in set(lens):
        cover = np.unique(np.concatenate([probed[b] for b, s in enumerate(seqs) if s.L == L]))
        assert np.array_equal(cover, st.edge_positions(L, split, s_q, prot)), f"edges of length {L} not all probed"
    print(f"{name} {mode}: {tried} mutated kernels, {tried - len(missed)} fail the checks", flush=True)
    assert not missed, f"{name} {mode}: mutations the checks do not see: {missed[:10]}"


RANDOM_BATCHES = [
    # (name, H, s_q, lens, c_bits, split) -- as in the GPU decode tests
    ("c4_h128_sq1_nosplit", 128, 1, [1, 31, 32, 33, 95, 200, 517], 4, 0),
    ("c4_h16_sq1_nosplit", 16, 1, [1, 7, 256, 333], 4, 0),
]


@pytest.mark.parametrize("batch", RANDOM_BATCHES, ids=[c[0] for c in RANDOM_BATCHES])
def test_dropped_key_in_random_batches_report(batch):
    name, H, s_q, lens, cb, split = batch
    w = syn.Workload(name, 999, B=len(lens), H=H, s_q=s_q, context=None, layers=((cb, 4),),
                     split_tokens=split, ctx_range=(1, 2))
    seqs = []
    for b, L in enumerate(lens):
        ctok, ktok = syn.sequence_tokens(w, 0, b, L)
        ql, qr = syn.queries(w, 0, batch=[b])
        c, k = oracle_values("lowbit", cb, "fp16", None, ctok, ktok)
        seqs.append(Sequence(ql[0], qr[0], c, k, s_q))
    exact = [s.exact() for s in seqs]
    AttnStats.merged(exact).check(f"{name} exact", quiet=True)
    seen = tried = 0
    rng = np.random.default_rng(1)
    for b, seq in enumerate(seqs):
        for p in rng.choice(seq.L, size=min(seq.L, 12), replace=False):
            out, lse = seq.mutated("drop", int(p))
            tried += 1
            try:
                AttnStats.merged(exact[:b] + exact[b + 1:] + [seq.stats(out, lse)]).check(quiet=True)
            except AssertionError:
                seen += 1
    print(f"{name}: a dropped key fails the checks in {seen} of {tried} random positions", flush=True)
    assert seen == tried

"""Offline-fusion identities of the two cache paths (CPU only, fp64, random weights).

Sec. 3.1 and Appendix C.1-C.2: weightless RMSNorm commutes with an orthogonal
rotation; the fused content cache ``z_C = u R_C S_C`` with compensated
consumers reproduces every consumer output; the reciprocal RoPE-pair
transform keeps the positional scores and commutes with RoPE at every
position (Proposition 1), so it folds into the pre-RoPE projections.  The
end-to-end check runs the oracle's absorbed decode attention on the fused
cache and fused queries: after the (fused) value projection the head outputs
equal the original ones, i.e. attention needs only the transformed latents.
Negative controls show what the constraints rule out: a rotation that mixes
frequency pairs does not commute with RoPE, and a non-reciprocal scale
changes the scores.
"""
import numpy as np
import pytest

from oracle import attention as at
from oracle import fusion as fu

D_C, D_R, D_MODEL, D_H = 64, 16, 96, 24


def _rng(k):
    return np.random.default_rng(1000 + k)


def test_weightless_rmsnorm_is_rotation_equivariant():
    rng = _rng(0)
    x = rng.standard_normal((50, D_C)) * 3
    R = fu.random_orthogonal(rng, D_C)
    np.testing.assert_allclose(fu.rmsnorm_weightless(x @ R), fu.rmsnorm_weightless(x) @ R, rtol=1e-12, atol=1e-12)
    # a non-orthogonal map breaks it
    A = R * rng.uniform(0.5, 2.0, D_C)[None, :]
    assert np.abs(fu.rmsnorm_weightless(x @ A) - fu.rmsnorm_weightless(x) @ A).max() > 1e-2


def test_content_fusion_preserves_every_consumer():
    rng = _rng(1)
    x = rng.standard_normal((40, D_MODEL))
    W_a = rng.standard_normal((D_MODEL, D_C)) / np.sqrt(D_MODEL)
    gamma = rng.uniform(0.2, 3.0, D_C)
    consumers = [rng.standard_normal((D_C, D_H)) for _ in range(3)]
    R_C = fu.random_orthogonal(rng, D_C)
    s_C = np.exp(rng.uniform(-1, 1, D_C))
    W_a2, gamma2, fused = fu.fuse_content(W_a, gamma, consumers, R_C, s_C)
    c = fu.content_latent(x @ W_a, gamma)
    z = fu.content_latent(x @ W_a2, gamma2)          # the fused cache, produced by the fused model
    np.testing.assert_allclose(z, fu.rmsnorm_weightless(x @ W_a) @ R_C * s_C[None, :], rtol=1e-11, atol=1e-12)
    for W_b, W_b2 in zip(consumers, fused):
        np.testing.assert_allclose(z @ W_b2, c @ W_b, rtol=1e-10, atol=1e-11)
    assert np.abs(z - c).max() > 0.1                  # the cache itself did change


def test_rope_reciprocal_transform_keeps_scores_and_commutes():
    rng = _rng(2)
    Q = rng.standard_normal((7, D_R))
    K = rng.standard_normal((30, D_R))
    ang = rng.uniform(-np.pi, np.pi, D_R // 2)
    sc = np.exp(rng.uniform(-1.5, 1.5, D_R // 2))
    RS = fu.pair_transform(ang, sc)
    RSi = fu.pair_transform(ang, 1.0 / sc)
    np.testing.assert_allclose((Q @ RSi) @ (K @ RS).T, Q @ K.T, rtol=1e-11, atol=1e-11)
    pos = rng.integers(0, 5000, 30)
    np.testing.assert_allclose(fu.apply_rope(K @ RS, pos), fu.apply_rope(K, pos) @ RS, rtol=1e-10, atol=1e-10)
    # negative controls: a rotation mixing frequency pairs, a non-reciprocal scale
    dense = fu.random_orthogonal(rng, D_R)
    assert np.abs(fu.apply_rope(K @ dense, pos) - fu.apply_rope(K, pos) @ dense).max() > 0.1
    assert np.abs((Q @ RS) @ (K @ RS).T - Q @ K.T).max() > 0.1


def test_fused_pre_rope_projections_keep_positional_scores():
    rng = _rng(3)
    hq = rng.standard_normal((5, D_MODEL))
    hk = rng.standard_normal((40, D_MODEL))
    W_Q = rng.standard_normal((D_MODEL, D_R)) / np.sqrt(D_MODEL)
    W_K = rng.standard_normal((D_MODEL, D_R)) / np.sqrt(D_MODEL)
    ang = rng.uniform(-np.pi, np.pi, D_R // 2)
    sc = np.exp(rng.uniform(-1, 1, D_R // 2))
    W_Q2, W_K2 = fu.fuse_rope(W_Q, W_K, ang, sc)
    qpos = np.full(5, 39)
    kpos = np.arange(40)
    want = fu.apply_rope(hq @ W_Q, qpos) @ fu.apply_rope(hk @ W_K, kpos).T
    got = fu.apply_rope(hq @ W_Q2, qpos) @ fu.apply_rope(hk @ W_K2, kpos).T
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("s_q", [1, 2])
def test_absorbed_decode_on_fused_cache_reproduces_head_outputs(s_q):
    """Full MLA decode with random weights: original vs fused model.

    Original: latent ``c`` cached, RoPE key ``k_r = RoPE(h W_KR)`` cached;
    per head, the absorbed content query is ``q_C W_UK^T`` and the output is
    ``softmax(tau (qbar c^T + q_R k_r^T)) c W_UV``.  Fused: cache ``z_C`` and
    the RoPE key from ``W_KR'``, queries from the fused projections; the same
    oracle attention over the fused cache, then the fused value projection.
    """
    rng = _rng(4 + s_q)
    H, L, tau = 4, 60, 1.0 / np.sqrt(D_H + D_R)
    x = rng.standard_normal((L, D_MODEL))
    W_a = rng.standard_normal((D_MODEL, D_C)) / np.sqrt(D_MODEL)
    gamma = rng.uniform(0.2, 3.0, D_C)
    W_UK = [rng.standard_normal((D_C, D_H)) / np.sqrt(D_C) for _ in range(H)]
    W_UV = [rng.standard_normal((D_C, D_H)) / np.sqrt(D_C) for _ in range(H)]
    W_KR = rng.standard_normal((D_MODEL, D_R)) / np.sqrt(D_MODEL)
    W_QR = [rng.standard_normal((D_MODEL, D_R)) / np.sqrt(D_MODEL) for _ in range(H)]
    W_QC = [rng.standard_normal((D_MODEL, D_H)) / np.sqrt(D_MODEL) for _ in range(H)]

    R_C = fu.random_orthogonal(rng, D_C)
    s_C = np.exp(rng.uniform(-1, 1, D_C))
    ang = rng.uniform(-np.pi, np.pi, D_R // 2)
    sc = np.exp(rng.uniform(-1, 1, D_R // 2))
    W_a2, gamma2, fused = fu.fuse_content(W_a, gamma, W_UK + W_UV, R_C, s_C)
    W_UK2, W_UV2 = fused[:H], fused[H:]
    W_QR2, W_KR2 = [], None
    for h in range(H):
        q2, k2 = fu.fuse_rope(W_QR[h], W_KR, ang, sc)
        W_QR2.append(q2)
        W_KR2 = k2

    pos = np.arange(L)
    qpos = pos[L - s_q:]
    hq = x[L - s_q:]

    def run(W_a_, gamma_, W_UK_, W_UV_, W_QR_, W_KR_):
        c = fu.content_latent(x @ W_a_, gamma_)            # the cache the model writes
        k_r = fu.apply_rope(x @ W_KR_, pos)
        outs = []
        for h in range(H):
            qbar = (hq @ W_QC[h]) @ W_UK_[h].T             # absorbed content query
            q_r = fu.apply_rope(hq @ W_QR_[h], qpos)
            lat, _ = at.attend(qbar, q_r, c, k_r, tau, at.decode_limits(L, s_q, 1))
            outs.append(lat @ W_UV_[h])
        return np.stack(outs), c

    want, c = run(W_a, gamma, W_UK, W_UV, W_QR, W_KR)
    got, z = run(W_a2, gamma2, W_UK2, W_UV2, W_QR2, W_KR2)
    np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-11)
    assert np.abs(z - c).max() > 0.1

"""Materialised (non-absorbed) MLA and the positional-QK bound -- oracle pins.

Sec. 2.1: per-head content keys and values are reconstructed from the latent
``C`` by up-projections; at inference the key up-projection is absorbed into
the query (``Qbar_C,h = Q_C,h W_K,h^T``) and the value projection moves past the
attention (``B_h``).  Computing a head the materialised way and comparing with
the absorbed form (followed by the value projection) pins ``attention.attend``
independently of its own arithmetic.

Sec. 3.2, Proposition 2 (proof in Appendix C.3): with content logits, queries,
values and valid key sets held fixed, a perturbation ``dZ_h`` of the unscaled
positional scores changes the head output by at most
``tau/2 * ||Omega . dZ_h||_F * ||Vbar_h||_2``.  In the latent space the kernel
returns, ``Vbar_h = C``.

Pure numpy, fp64; shares no code with the GPU library.
"""
from __future__ import annotations

import math

import numpy as np


def materialised_head(q_nope, q_rope, c, k_rope, w_uk, w_uv, tau, limits):
    """One head computed with explicit per-head keys and values.

    ``q_nope [R, d_h]``, ``q_rope [R, d_r]``, latent ``c [L, d_c]``, RoPE key
    ``k_rope [L, d_r]``, up-projections ``w_uk [d_c, d_h]``, ``w_uv [d_c, d_v]``.
    Row ``r`` attends to keys ``t < limits[r]``.  Returns ``[R, d_v]``.
    """
    keys = np.asarray(c, np.float64) @ np.asarray(w_uk, np.float64)      # [L, d_h]
    vals = np.asarray(c, np.float64) @ np.asarray(w_uv, np.float64)      # [L, d_v]
    out = np.zeros((len(q_nope), vals.shape[1]))
    for r in range(len(q_nope)):
        n = int(limits[r])
        sc = [tau * (float(np.dot(q_nope[r], keys[t])) + float(np.dot(q_rope[r], k_rope[t])))
              for t in range(n)]
        mx = max(sc)
        w = [math.exp(v - mx) for v in sc]
        tot = math.fsum(w)
        out[r] = sum((wi / tot) * vals[t] for t, wi in enumerate(w))
    return out


def brute_force_rows(q_lat, q_rope, c_hat, kr_hat, tau, limits):
    """Scalar-loop attention (lists and ``math`` only) for tiny inputs.

    Returns ``(out, lse)`` as nested Python lists; an independent restatement
    of the softmax definition used to pin ``attention.attend``.
    """
    outs, lses = [], []
    d_c = len(c_hat[0])
    for r in range(len(q_lat)):
        z = []
        for t in range(int(limits[r])):
            acc = math.fsum(float(q_lat[r][c]) * float(c_hat[t][c]) for c in range(d_c))
            acc += math.fsum(float(q_rope[r][c]) * float(kr_hat[t][c]) for c in range(len(kr_hat[t])))
            z.append(tau * acc)
        mx = max(z)
        den = math.fsum(math.exp(v - mx) for v in z)
        row = [math.fsum(math.exp(z[t] - mx) * float(c_hat[t][c]) for t in range(len(z))) / den
               for c in range(d_c)]
        outs.append(row)
        lses.append(mx + math.log(den))
    return outs, lses


def positional_bound(tau, dz_masked, c):
    """Right-hand side of Proposition 2 for one head with ``Vbar_h = C``.

    ``dz_masked`` is the unscaled positional-score perturbation with invalid
    pairs already zeroed; ``c`` the latent rows the head attends to.
    """
    return 0.5 * tau * np.linalg.norm(dz_masked, 'fro') * np.linalg.norm(np.asarray(c, np.float64), 2)

"""Closed forms that pin the oracle (test infrastructure only).

Neither function reuses the oracle's loop; each writes the result of the
recurrence in a different, textbook form so that a dropped term, a wrong sign
or a transposed operand in the oracle shows up as a mismatch.

* ``unrolled_states``: the recurrence of Eq. (gdn) (paper Sec. 4.1) with scalar
  gates, unrolled into explicit d_k x d_k transition matrices
      M_s = (I - b_s k_s k_s^T) exp(g_s),
      S_t = (M_t ... M_1) S_0 + sum_{s<=t} (M_t ... M_{s+1}) w_s k_s v_s^T,
  built from full matrix products (no rank-one updates).
* ``decay_attention``: the scalar-decay member (b = 0, w = 1) written as dense
  masked, decayed attention over the whole sequence,
      O = ((Q K^T) * D) V + diag(exp(G)) Q S_0,  D_ts = exp(G_t - G_s) for s <= t,
  with G the cumulative sum of g over the whole sequence (an O(L^2) form).
"""
from __future__ import annotations

import numpy as np


def unrolled_states(k, v, g, b, w, S0):
    """One stream: k [L,dk], v [L,dv], g, b, w [L], S0 [dk,dv] -> S_t for t=0..L (S_0 first)."""
    L, dk = k.shape
    I = np.eye(dk)
    M = [(I - b[s] * np.outer(k[s], k[s])) * np.exp(g[s]) for s in range(L)]
    out = [S0.copy()]
    for t in range(1, L + 1):
        prod = np.eye(dk)
        for s in range(t - 1, -1, -1):  # prod = M_t ... M_1 (0-based M[t-1] ... M[0])
            prod = prod @ M[s]
        S = prod @ S0
        for s in range(t):
            tail = np.eye(dk)
            for r in range(t - 1, s, -1):  # M_t ... M_{s+1}
                tail = tail @ M[r]
            S = S + tail @ (w[s] * np.outer(k[s], v[s]))
        out.append(S)
    return out


def decay_attention(q, k, v, g, S0):
    """One stream of the scalar-decay member: returns O [L,dv] and S_T."""
    L = q.shape[0]
    G = np.cumsum(g)
    t_idx = np.arange(L)
    mask = t_idx[:, None] >= t_idx[None, :]
    D = np.where(mask, np.exp(np.where(mask, G[:, None] - G[None, :], 0.0)), 0.0)
    O = ((q @ k.T) * D) @ v + np.exp(G)[:, None] * (q @ S0)
    S_T = np.exp(G[-1]) * S0 + (np.exp(G[-1] - G)[:, None] * k).T @ v
    return O, S_T


__all__ = ["unrolled_states", "decay_attention"]

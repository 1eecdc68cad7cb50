"""Chunked float64 reference of the gated delta rule (forward and backward).

TEST INFRASTRUCTURE ONLY (same rules as ``gdn_oracle``).  It shares no code
with the HIP path and none with the token-serial oracle either: it is the
chunkwise rung of the paper's reference ladder (Sec. 4.5), checked against the
token-serial oracle, which sits below it.

One stream at a time (2-D arrays), any chunk size C (the last chunk may hold
C' < C tokens).  Within a chunk, with r, i the positions 1..C':

  G_r = sum_{s<=r} g_s (in-chunk cumulative log-decay),  Gam_r = exp(G_r)
  D_ri = exp(G_r - G_i) for i <= r, else 0    (the exponent is formed only where
                                                i <= r: select, then exp; paper
                                                Sec. 4.5, masked-exp fix)
  A   = strictly-lower( diag(b) (K K^T) * D )             erase coupling
  T   = (I + A)^{-1}                                      (Sec. 4.2, K#2)
  W   = T diag(b * Gam) K,   U = T diag(w) V              (the two applies)
  U'  = U - W h                                           corrected values
  O   = diag(Gam) Q h + ((Q K^T) * D) U'                  chunk output
  h  <- Gam_{C'} h + Khat^T U',  Khat_r = exp(G_{C'} - G_r) k_r   (carry)

with b = w = beta for the delta-rule variants and b = 0, w = 1 for the
scalar-decay variant (the family table's gate settings), where A = 0 and T = I.

T is computed by forward substitution, which is the definition of the inverse
of a unit lower-triangular matrix: row r of T is e_r - sum_{i<r} A_ri T_i.

The backward walks the chunks in reverse with the carry dh (the K#1 reverse
state scan) and differentiates each chunk's steps in reverse (the K#2 VJP of
the solve reuses T: dA = -T^T dT T^T restricted to the strict lower triangle).
The dg of a chunk is the reverse cumulative sum of dG over the chunk.
"""
from __future__ import annotations

import numpy as np

VARIANTS = ("gated_delta", "delta", "decay_only")


def _f64(x):
    if x is not None and (not isinstance(x, np.ndarray) or x.dtype != np.float64):
        raise TypeError("chunked reference takes float64 arrays only")
    return x


def forward_substitution_inverse(A: np.ndarray) -> np.ndarray:
    """(I + A)^{-1} for strictly lower-triangular A, row by row."""
    n = A.shape[0]
    T = np.zeros_like(A)
    for r in range(n):
        row = np.zeros(n)
        row[r] = 1.0
        for i in range(r):
            row -= A[r, i] * T[i]
        T[r] = row
    return T


def _gates(variant, g, beta, t0, t1):
    n = t1 - t0
    gg = np.zeros(n) if variant == "delta" else g[t0:t1]
    if variant == "decay_only":
        b, w = np.zeros(n), np.ones(n)
    else:
        b = beta[t0:t1]
        w = b
    return gg, b, w


def _chunk_fwd(Q, K, V, gg, b, w, h):
    n = Q.shape[0]
    G = np.cumsum(gg)
    Gam = np.exp(G)
    low = np.tril(np.ones((n, n), dtype=bool))
    diff = np.where(low, G[:, None] - G[None, :], 0.0)
    D = np.where(low, np.exp(diff), 0.0)
    Bm = K @ K.T
    A = np.tril(b[:, None] * Bm * D, -1)
    T = forward_substitution_inverse(A)
    Kb = (b * Gam)[:, None] * K
    Vw = w[:, None] * V
    W = T @ Kb
    U = T @ Vw
    Up = U - W @ h
    QK = Q @ K.T
    P = QK * D
    O = Gam[:, None] * (Q @ h) + P @ Up
    decay_to_end = np.exp(G[-1] - G)
    Khat = decay_to_end[:, None] * K
    h_next = Gam[-1] * h + Khat.T @ Up
    return dict(G=G, Gam=Gam, D=D, Bm=Bm, A=A, T=T, Kb=Kb, Vw=Vw, W=W, U=U, Up=Up, QK=QK, P=P,
                O=O, Khat=Khat, decay_to_end=decay_to_end, h=h, h_next=h_next)


def chunked_fwd(q, k, v, g, beta, S0, variant="gated_delta", C=64, keep=False):
    """One stream: q, k [L,dk]; v [L,dv]; g, beta [L]; S0 [dk,dv].

    Returns (o, S_T, chunk_states[NT,dk,dv]) and, with keep=True, the list of
    per-chunk intermediates as a fourth item.
    """
    for x in (q, k, v, g, beta, S0):
        _f64(x)
    if variant not in VARIANTS:
        raise ValueError(variant)
    L, dk = q.shape
    dv = v.shape[1]
    h = S0.copy()
    o = np.zeros((L, dv))
    states, inter = [], []
    for t0 in range(0, L, C):
        t1 = min(L, t0 + C)
        gg, b, w = _gates(variant, g, beta, t0, t1)
        st = _chunk_fwd(q[t0:t1], k[t0:t1], v[t0:t1], gg, b, w, h)
        states.append(h)
        o[t0:t1] = st["O"]
        h = st["h_next"]
        if keep:
            inter.append(st)
    states = np.array(states).reshape(-1, dk, dv)
    return (o, h, states, inter) if keep else (o, h, states)


def _chunk_bwd(Q, K, V, st, b, w, dO, dh, variant):
    """Backward of one chunk.  Returns (dQ, dK, dV, dG, db, dw, dh_prev, dUp)."""
    G, Gam, D, Bm, A, T = st["G"], st["Gam"], st["D"], st["Bm"], st["A"], st["T"]
    Kb, Vw, W, Up, P, Khat, h = st["Kb"], st["Vw"], st["W"], st["Up"], st["P"], st["Khat"], st["h"]
    dte = st["decay_to_end"]
    # reverse state step and the gradient of the corrected values
    dUp = P.T @ dO + Khat @ dh
    dh_prev = Gam[-1] * dh + Q.T @ (Gam[:, None] * dO) - W.T @ dUp
    # output products
    dP = dO @ Up.T
    dPm = dP * D
    dQ = dPm @ K + Gam[:, None] * (dO @ h.T)
    dK = dPm.T @ Q
    dKhat = Up @ dh.T
    dK = dK + dte[:, None] * dKhat
    dW = -dUp @ h.T
    # the two applies U = T Vw, W = T Kb
    Y = T.T @ dUp
    X = T.T @ dW
    dV = w[:, None] * Y
    dw = np.sum(V * Y, axis=1)
    dK = dK + (b * Gam)[:, None] * X
    kx = np.sum(K * X, axis=1)
    db = Gam * kx
    dGam = b * kx
    # the solve T = (I + A)^{-1}
    dT = dUp @ Vw.T + dW @ Kb.T
    dA = np.tril(-(T.T @ dT @ T.T), -1)
    dBm = dA * b[:, None] * D
    db = db + np.sum(dA * Bm * D, axis=1)
    dK = dK + (dBm + dBm.T) @ K
    # decay masks and gains
    Z = dA * A + dP * P
    dG = Z.sum(axis=1) - Z.sum(axis=0)
    dGam = dGam + np.sum(dO * (Q @ h), axis=1)
    dG = dG + Gam * dGam
    kk = np.sum(Khat * dKhat, axis=1)
    dG = dG - kk
    dG[-1] += Gam[-1] * np.sum(h * dh) + kk.sum()
    return dQ, dK, dV, dG, db, dw, dh_prev, dUp


def chunked_bwd(q, k, v, g, beta, S0, dO, dS_T, variant="gated_delta", C=64, keep=False):
    """One stream.  Returns (dq, dk, dv, dg, dbeta, dS0) (+ per-chunk dh, dUp with keep)."""
    for x in (q, k, v, g, beta, S0, dO, dS_T):
        _f64(x)
    L, dk = q.shape
    dv = v.shape[1]
    _, _, _, inter = chunked_fwd(q, k, v, g, beta, S0, variant, C, keep=True)
    dq, dk_, dvv = np.zeros((L, dk)), np.zeros((L, dk)), np.zeros((L, dv))
    dg = None if variant == "delta" else np.zeros(L)
    db = None if variant == "decay_only" else np.zeros(L)
    dh = dS_T.copy()
    saved = []
    starts = list(range(0, L, C))
    for c in range(len(starts) - 1, -1, -1):
        t0 = starts[c]
        t1 = min(L, t0 + C)
        _, b, w = _gates(variant, g, beta, t0, t1)
        dh_next = dh
        dQ, dK, dV, dG, dbb, dww, dh, dUp = _chunk_bwd(q[t0:t1], k[t0:t1], v[t0:t1], inter[c], b,
                                                       w, dO[t0:t1], dh_next, variant)
        dq[t0:t1], dk_[t0:t1], dvv[t0:t1] = dQ, dK, dV
        if dg is not None:
            dg[t0:t1] = np.cumsum(dG[::-1])[::-1]
        if db is not None:
            db[t0:t1] = dbb + dww
        if keep:
            saved.append(dict(dh_next=dh_next, dUp=dUp))
    out = (dq, dk_, dvv, dg, db, dh)
    return out + (saved[::-1],) if keep else out


__all__ = ["forward_substitution_inverse", "chunked_fwd", "chunked_bwd"]

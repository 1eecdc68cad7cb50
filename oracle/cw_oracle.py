"""Token-serial float64 oracle of the general (channel-wise) recurrence and its adjoint.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this module.  It shares no code with the HIP
path: a plain, slow loop over tokens.

What it computes: the paper's general recurrence (Sec. 4.1, Eq. (gdn)) with its
three gates per channel,

    S_t = (I - k_t (b_t * k_t)^T) Diag(e^{g_t}) S_{t-1} + k_t (w_t * v_t)^T,
    o_t = S_t^T q_t,

for one stream (one sequence, one head), S of shape d_k x d_v; g_t (log-decay)
and b_t (erase) have d_k entries, w_t (write) has d_v.  A missing gate takes
its neutral value: g = 0, b = 0 (no erase), w = 1.  The family table's
members are gate settings: KDA is b = w = beta_t (a scalar per token),
GLA is b = 0, w = 1, LA additionally g = 0.

The loop performs, per token (the grouping is the algorithm's; no fusion):

    St = e^{g_t} (row-scaled: row d of S times e^{g_t[d]})
    p  = St^T (b_t * k_t)                  (d_v)
    u  = w_t * v_t - p
    S_t = St + k_t u^T
    o_t = S_t^T q_t

Backward, for the loss sum(dO * o) + <dS_T, S_T>, hand-derived by reverse-mode
through the steps above, t = L-1 down to 0:

    dS  += q_t dO_t^T;        dq_t = S_t dO_t
    du   = dS^T k_t;          dk_t = dS u
    dv_t = w_t * du;          dw_t = v_t * du
    dp   = -du
    dSt  = dS + (b_t * k_t) dp^T
    dkb  = St dp;             dk_t += b_t * dkb;   db_t = k_t * dkb
    dg_t = rowsum(dSt * St)   (d_k: the derivative through e^{g_t[d]})
    dS   = e^{g_t} * dSt      (row-scaled)

and dS0 = dS at the end.  A chunk's states are recomputed from its checkpoint
(chunk_states[c] = the state before token c * chunk), so memory stays
O(chunk * d_k * d_v).

Every array must be float64 (complex128 is accepted for the complex-step
derivative check).
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

_OK_DTYPES = (np.dtype(np.float64), np.dtype(np.complex128))


def _need(x, name):
    if x is None:
        return None
    if not isinstance(x, np.ndarray) or x.dtype not in _OK_DTYPES:
        raise TypeError(f"oracle: {name} must be a float64 (or complex128) ndarray, got "
                        f"{getattr(x, 'dtype', type(x))}")
    return x


# --------------------------------------------------------------------------
# Stream-batched cores: q, k [NS, L, dk]; v, dO [NS, L, dv]; g, b [NS, L, dk];
# w [NS, L, dv]; S0, dS_T [NS, dk, dv].  g, b, w may be None.
# --------------------------------------------------------------------------

def _step(S, k_t, v_t, g_t, b_t, w_t):
    """One token: returns (St, kb, u, S_new)."""
    St = S if g_t is None else np.exp(g_t)[:, :, None] * S
    wv = v_t if w_t is None else w_t * v_t
    if b_t is None:
        kb = None
        u = wv
    else:
        kb = b_t * k_t
        u = wv - np.einsum("skv,sk->sv", St, kb)
    S_new = St + k_t[:, :, None] * u[:, None, :]
    return St, kb, u, S_new


def cw_fwd_streams(q, k, v, g, b, w, S0, chunk=64):
    """Token-serial forward.  Returns (o [NS,L,dv], S_T [NS,dk,dv], chunk_states [NS,NT,dk,dv])."""
    for name, x in (("q", q), ("k", k), ("v", v), ("g", g), ("b", b), ("w", w), ("S0", S0)):
        _need(x, name)
    NS, L, dk = q.shape
    dv = v.shape[-1]
    dt = np.result_type(q, k, v, S0, *(x for x in (g, b, w) if x is not None))
    NT = -(-L // chunk)
    o = np.zeros((NS, L, dv), dt)
    states = np.zeros((NS, NT, dk, dv), dt)
    S = np.array(S0, dtype=dt, copy=True)
    for t in range(L):
        if t % chunk == 0:
            states[:, t // chunk] = S
        _, _, _, S = _step(S, k[:, t], v[:, t], None if g is None else g[:, t],
                           None if b is None else b[:, t], None if w is None else w[:, t])
        o[:, t] = np.einsum("skv,sk->sv", S, q[:, t])
    return o, S, states


def cw_bwd_streams(q, k, v, g, b, w, S0, dO, dS_T, chunk=64):
    """Token-serial adjoint.  Returns (dq, dk, dv, dg, db, dw, dS0); a gate's
    gradient is None when the gate is None."""
    for name, x in (("q", q), ("k", k), ("v", v), ("g", g), ("b", b), ("w", w), ("S0", S0),
                    ("dO", dO), ("dS_T", dS_T)):
        _need(x, name)
    NS, L, dk = q.shape
    dv_ = v.shape[-1]
    dt = np.result_type(q, k, v, S0, dO, dS_T, *(x for x in (g, b, w) if x is not None))
    _, _, states = cw_fwd_streams(q, k, v, g, b, w, S0, chunk)
    NT = states.shape[1]
    dq = np.zeros((NS, L, dk), dt)
    dk_ = np.zeros((NS, L, dk), dt)
    dvv = np.zeros((NS, L, dv_), dt)
    dg = None if g is None else np.zeros((NS, L, dk), dt)
    db = None if b is None else np.zeros((NS, L, dk), dt)
    dw = None if w is None else np.zeros((NS, L, dv_), dt)
    dS = np.array(dS_T, dtype=dt, copy=True)
    for c in range(NT - 1, -1, -1):
        t0, t1 = c * chunk, min(L, (c + 1) * chunk)
        S = states[:, c]
        rec = []
        for t in range(t0, t1):
            St, kb, u, S = _step(S, k[:, t], v[:, t], None if g is None else g[:, t],
                                 None if b is None else b[:, t], None if w is None else w[:, t])
            rec.append((St, kb, u, S))
        for t in range(t1 - 1, t0 - 1, -1):
            St, kb, u, S_t = rec[t - t0]
            k_t, q_t, do_t = k[:, t], q[:, t], dO[:, t]
            dS = dS + q_t[:, :, None] * do_t[:, None, :]
            dq[:, t] = np.einsum("skv,sv->sk", S_t, do_t)
            du = np.einsum("skv,sk->sv", dS, k_t)
            dkt = np.einsum("skv,sv->sk", dS, u)
            dvv[:, t] = du if w is None else w[:, t] * du
            if w is not None:
                dw[:, t] = v[:, t] * du
            if b is None:
                dSt = dS
            else:
                dp = -du
                dSt = dS + kb[:, :, None] * dp[:, None, :]
                dkb = np.einsum("skv,sv->sk", St, dp)
                dkt = dkt + b[:, t] * dkb
                db[:, t] = k_t * dkb
            dk_[:, t] = dkt
            if g is None:
                dS = dSt
            else:
                dg[:, t] = np.einsum("skv,skv->sk", dSt, St)
                dS = np.exp(g[:, t])[:, :, None] * dSt
    return dq, dk_, dvv, dg, db, dw, dS


# --------------------------------------------------------------------------
# Layout-level entry points: q, k, g, b [B,T,H,dk]; v, w, dO [B,T,H,dv];
# S0, dS_T [N,H,dk,dv]; optional cu_seqlens (packed sequences, B = 1).
# --------------------------------------------------------------------------

def _seq_slices(B, T, cu_seqlens):
    if cu_seqlens is None:
        return [(bb, 0, T) for bb in range(B)]
    if B != 1:
        raise ValueError("packed sequences need B == 1")
    cu = [int(x) for x in cu_seqlens]
    return [(0, cu[n], cu[n + 1] - cu[n]) for n in range(len(cu) - 1)]


def _gather(x, bb, s, L):
    """[B,T,H,...] -> [H, L, ...] for one sequence."""
    return None if x is None else np.moveaxis(x[bb, s:s + L], 1, 0)


def cw_oracle_fwd(q, k, v, g, b, w, S0, *, cu_seqlens=None, chunk=64,
                  heads: Optional[Sequence[int]] = None):
    """Forward over the API layout.  Returns (o, S_T, chunk_states); chunk_states
    is [sum_n ceil(L_n/chunk), H, dk, dv].  Heads outside ``heads`` stay NaN."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    seqs = _seq_slices(B, T, cu_seqlens)
    N = len(seqs)
    if S0 is None:
        S0 = np.zeros((N, H, dk, dv))
    hs = list(range(H)) if heads is None else list(heads)
    nt = [-(-L // chunk) for (_, _, L) in seqs]
    off = np.concatenate([[0], np.cumsum(nt)]).astype(int)
    o = np.full((B, T, H, dv), np.nan)
    S_T = np.full((N, H, dk, dv), np.nan)
    states = np.full((int(off[-1]), H, dk, dv), np.nan)
    for n, (bb, s, L) in enumerate(seqs):
        sub = lambda x: None if x is None else _gather(x, bb, s, L)[hs]
        o_n, ST_n, st_n = cw_fwd_streams(sub(q), sub(k), sub(v), sub(g), sub(b), sub(w), S0[n, hs], chunk)
        o[bb, s:s + L][:, hs] = np.moveaxis(o_n, 0, 1)
        S_T[n, hs] = ST_n
        states[off[n]:off[n + 1], hs] = np.moveaxis(st_n, 0, 1)
    return o, S_T, states


def cw_oracle_bwd(q, k, v, g, b, w, S0, dO, dS_T, *, cu_seqlens=None, chunk=64,
                  heads: Optional[Sequence[int]] = None):
    """Backward over the API layout.  Returns (dq, dk, dv, dg, db, dw, dS0)."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    seqs = _seq_slices(B, T, cu_seqlens)
    N = len(seqs)
    if S0 is None:
        S0 = np.zeros((N, H, dk, dv))
    if dS_T is None:
        dS_T = np.zeros((N, H, dk, dv))
    hs = list(range(H)) if heads is None else list(heads)
    full = lambda like, last: None if like is None else np.full((B, T, H, last), np.nan)
    dq, dk_, dvv = full(q, dk), full(k, dk), full(v, dv)
    dg, db, dw = full(g, dk), full(b, dk), full(w, dv)
    dS0 = np.full((N, H, dk, dv), np.nan)
    for n, (bb, s, L) in enumerate(seqs):
        sub = lambda x: None if x is None else _gather(x, bb, s, L)[hs]
        r = cw_bwd_streams(sub(q), sub(k), sub(v), sub(g), sub(b), sub(w), S0[n, hs], sub(dO),
                           dS_T[n, hs], chunk)
        for out, res in zip((dq, dk_, dvv, dg, db, dw), r[:6]):
            if out is not None:
                out[bb, s:s + L][:, hs] = np.moveaxis(res, 0, 1)
        dS0[n, hs] = r[6]
    return dq, dk_, dvv, dg, db, dw, dS0


__all__ = ["cw_fwd_streams", "cw_bwd_streams", "cw_oracle_fwd", "cw_oracle_bwd"]

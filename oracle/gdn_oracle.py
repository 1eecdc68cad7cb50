"""Token-serial float64 oracle of the gated delta rule and its hand-derived adjoint.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this module.  It shares no code with the HIP
path: it is a plain, slow, obviously correct loop over tokens.

What it computes (paper Sec. 4.1, Eq. (gdn), scalar gates b = w = beta and a
scalar log-decay g; this is the KDA row of the family table with a scalar gate,
which is what the path implements).  Per stream (one sequence, one head), with
S of shape d_k x d_v:

    S_t = (I - beta_t k_t k_t^T) e^{g_t} S_{t-1} + beta_t k_t v_t^T,   o_t = S_t^T q_t.

Written as the operations the loop performs (the grouping fixes which entries
become NaN/Inf when an input is non-finite):

    St = gamma_t * S_{t-1}                  gamma_t = exp(g_t)
    p  = St^T k_t                           (d_v)
    u  = beta_t * (v_t - p)
    S_t = St + k_t u^T
    o_t = S_t^T q_t

Family members (paper, table "One recurrence, five models"):
  * "gated_delta": the recurrence above.
  * "delta"      : DeltaNet, g identically 0 (gamma = 1, no multiply, no dg).
  * "decay_only" : the scalar-decay SSD / Mamba-2 row, b = 0 and w = 1, so
                   u = v_t and there is no beta.

Chunk states: chunk_states[c] is the state before token c*chunk of the stream
(so chunk_states[0] = S0), one per chunk of ``chunk`` tokens, ceil(L/chunk) of
them.  The sequential carry between chunks is the paper's chunking (Sec. 4.2).

Backward: the reverse-time adjoint of the loop above, differentiated by hand,
for the loss  sum(dO * o) + <dS_T, S_T>.  For t = L-1 down to 0:

    dS  += q_t dO_t^T;         dq_t = S_t dO_t
    du   = dS^T k_t;           dk_t = dS u
    (delta rule)  dbeta_t = du . (v_t - p);  dv_t = beta_t du;  dp = -beta_t du
                  dSt = dS + k_t dp^T;       dk_t += St dp
    (decay_only)  dv_t = du;  dSt = dS
    dg_t = <dSt, St>_F  (absent for "delta")
    dS   = gamma_t * dSt
and dS0 = dS at the end.  The states S_{t-1}, St, p, u, S_t of a chunk are
recomputed from that chunk's checkpoint, so memory stays O(chunk * d_k * d_v).

The oracle refuses reduced precision (paper Sec. 3.1: the reference runs in
full precision only): every array must be float64, or complex128 for the
complex-step derivative check.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

VARIANTS = ("gated_delta", "delta", "decay_only")
_OK_DTYPES = (np.dtype(np.float64), np.dtype(np.complex128))


def _need(x, name):
    if x is None:
        return None
    if not isinstance(x, np.ndarray) or x.dtype not in _OK_DTYPES:
        raise TypeError(f"oracle: {name} must be a float64 (or complex128) ndarray, got "
                        f"{getattr(x, 'dtype', type(x))}")
    return x


def _check_variant(variant, g, beta):
    if variant not in VARIANTS:
        raise ValueError(f"unknown variant {variant!r}")
    if variant != "delta" and g is None:
        raise ValueError("g is required for this variant")
    if variant != "decay_only" and beta is None:
        raise ValueError("beta is required for this variant")


# --------------------------------------------------------------------------
# Stream-batched cores.  Arrays carry a leading axis of independent streams:
# q, k [NS, L, dk]; v, dO [NS, L, dv]; g, beta [NS, L]; S0, dS_T [NS, dk, dv].
# --------------------------------------------------------------------------

def _step_fwd(S, k_t, v_t, g_t, b_t, variant):
    """One token: returns (St, p, u, S_new).  p is None without the delta term."""
    if variant == "delta":
        St = S
    else:
        St = np.exp(g_t)[:, None, None] * S
    if variant == "decay_only":
        p = None
        u = v_t
    else:
        p = np.einsum("skv,sk->sv", St, k_t)
        u = b_t[:, None] * (v_t - p)
    S_new = St + k_t[:, :, None] * u[:, None, :]
    return St, p, u, S_new


def fwd_streams(q, k, v, g, beta, S0, variant="gated_delta", chunk=64):
    """Token-serial forward over a batch of independent streams.

    Returns (o [NS,L,dv], S_T [NS,dk,dv], chunk_states [NS,NT,dk,dv]).
    """
    for name, x in (("q", q), ("k", k), ("v", v), ("g", g), ("beta", beta), ("S0", S0)):
        _need(x, name)
    _check_variant(variant, g, beta)
    NS, L, dk = q.shape
    dv = v.shape[-1]
    dt = np.result_type(q, k, v, S0, *(x for x in (g, beta) if x is not None))
    NT = -(-L // chunk)
    o = np.zeros((NS, L, dv), dt)
    states = np.zeros((NS, NT, dk, dv), dt)
    S = np.array(S0, dtype=dt, copy=True)
    for t in range(L):
        if t % chunk == 0:
            states[:, t // chunk] = S
        g_t = None if g is None else g[:, t]
        b_t = None if beta is None else beta[:, t]
        _, _, _, S = _step_fwd(S, k[:, t], v[:, t], g_t, b_t, variant)
        o[:, t] = np.einsum("skv,sk->sv", S, q[:, t])
    return o, S, states


def bwd_streams(q, k, v, g, beta, S0, dO, dS_T, variant="gated_delta", chunk=64):
    """Token-serial adjoint over a batch of independent streams.

    Returns (dq, dk, dv, dg, dbeta, dS0); dg is None for "delta" and dbeta is
    None for "decay_only".
    """
    for name, x in (("q", q), ("k", k), ("v", v), ("g", g), ("beta", beta), ("S0", S0),
                    ("dO", dO), ("dS_T", dS_T)):
        _need(x, name)
    _check_variant(variant, g, beta)
    NS, L, dk = q.shape
    dv_ = v.shape[-1]
    dt = np.result_type(q, k, v, S0, dO, dS_T, *(x for x in (g, beta) if x is not None))
    _, _, states = fwd_streams(q, k, v, g, beta, S0, variant, chunk)
    NT = states.shape[1]

    dq = np.zeros((NS, L, dk), dt)
    dk_ = np.zeros((NS, L, dk), dt)
    dvv = np.zeros((NS, L, dv_), dt)
    dg = None if variant == "delta" else np.zeros((NS, L), dt)
    db = None if variant == "decay_only" else np.zeros((NS, L), dt)
    dS = np.array(dS_T, dtype=dt, copy=True)

    for c in range(NT - 1, -1, -1):
        t0, t1 = c * chunk, min(L, (c + 1) * chunk)
        # Recompute the chunk's forward from its checkpoint.
        S = states[:, c]
        rec = []
        for t in range(t0, t1):
            g_t = None if g is None else g[:, t]
            b_t = None if beta is None else beta[:, t]
            St, p, u, S = _step_fwd(S, k[:, t], v[:, t], g_t, b_t, variant)
            rec.append((St, p, u, S))
        for t in range(t1 - 1, t0 - 1, -1):
            St, p, u, S_t = rec[t - t0]
            k_t, q_t, do_t = k[:, t], q[:, t], dO[:, t]
            dS = dS + q_t[:, :, None] * do_t[:, None, :]
            dq[:, t] = np.einsum("skv,sv->sk", S_t, do_t)
            du = np.einsum("skv,sk->sv", dS, k_t)
            dkt = np.einsum("skv,sv->sk", dS, u)
            if variant == "decay_only":
                dvv[:, t] = du
                dSt = dS
            else:
                b_t = beta[:, t]
                db[:, t] = np.einsum("sv,sv->s", du, v[:, t] - p)
                dvv[:, t] = b_t[:, None] * du
                dp = -b_t[:, None] * du
                dSt = dS + k_t[:, :, None] * dp[:, None, :]
                dkt = dkt + np.einsum("skv,sv->sk", St, dp)
            dk_[:, t] = dkt
            if variant == "delta":
                dS = dSt
            else:
                dg[:, t] = np.einsum("skv,skv->s", dSt, St)
                dS = np.exp(g[:, t])[:, None, None] * dSt
    return dq, dk_, dvv, dg, db, dS


# --------------------------------------------------------------------------
# Layout-level entry points: q, k [B,T,H,dk]; v, dO [B,T,H,dv]; g, beta [B,T,H];
# S0, dS_T [N,H,dk,dv]; optional cu_seqlens (packed sequences, B = 1).
# --------------------------------------------------------------------------

def _seq_slices(B, T, cu_seqlens):
    if cu_seqlens is None:
        return [(b, 0, T) for b in range(B)]
    if B != 1:
        raise ValueError("packed sequences need B == 1")
    cu = [int(x) for x in cu_seqlens]
    return [(0, cu[n], cu[n + 1] - cu[n]) for n in range(len(cu) - 1)]


def _gather(x, b, s, L):
    """[B,T,H,...] -> [H, L, ...] for one sequence."""
    if x is None:
        return None
    return np.moveaxis(x[b, s:s + L], 1, 0)


def _group_size(H, dk, dv, chunk, budget_bytes=1 << 28):
    per_stream = (chunk + 4) * dk * dv * 8 * 4
    return max(1, min(H, budget_bytes // max(per_stream, 1)))


def oracle_fwd(q, k, v, g, beta, S0, *, variant="gated_delta", cu_seqlens=None, chunk=64,
               heads: Optional[Sequence[int]] = None):
    """Forward over the API layout.  Returns (o, S_T, chunk_states).

    chunk_states is [sum_n ceil(L_n/chunk), H, dk, dv] with sequence n's chunks
    at offsets sum_{m<n} ceil(L_m/chunk).  ``heads`` restricts the work to a
    subset of heads (other entries are left as NaN) for sampled checks.
    """
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
    grp = _group_size(len(hs), dk, dv, chunk)
    for n, (b, s, L) in enumerate(seqs):
        for i in range(0, len(hs), grp):
            hh = hs[i:i + grp]
            sub = lambda x: None if x is None else _gather(x, b, s, L)[hh]
            o_n, ST_n, st_n = fwd_streams(sub(q), sub(k), sub(v), sub(g), sub(beta),
                                          S0[n, hh], variant, chunk)
            o[b, s:s + L][:, hh] = np.moveaxis(o_n, 0, 1)
            S_T[n, hh] = ST_n
            states[off[n]:off[n + 1], hh] = np.moveaxis(st_n, 0, 1)
    return o, S_T, states


def oracle_bwd(q, k, v, g, beta, S0, dO, dS_T, *, variant="gated_delta", cu_seqlens=None,
               chunk=64, heads: Optional[Sequence[int]] = None):
    """Backward over the API layout.  Returns (dq, dk, dv, dg, dbeta, dS0)."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    seqs = _seq_slices(B, T, cu_seqlens)
    N = len(seqs)
    if S0 is None:
        S0 = np.zeros((N, H, dk, dv))
    if dS_T is None:
        dS_T = np.zeros((N, H, dk, dv))
    hs = list(range(H)) if heads is None else list(heads)
    dq = np.full((B, T, H, dk), np.nan)
    dk_ = np.full((B, T, H, dk), np.nan)
    dvv = np.full((B, T, H, dv), np.nan)
    dg = None if variant == "delta" else np.full((B, T, H), np.nan)
    db = None if variant == "decay_only" else np.full((B, T, H), np.nan)
    dS0 = np.full((N, H, dk, dv), np.nan)
    grp = _group_size(len(hs), dk, dv, chunk)
    for n, (b, s, L) in enumerate(seqs):
        for i in range(0, len(hs), grp):
            hh = hs[i:i + grp]
            sub = lambda x: None if x is None else _gather(x, b, s, L)[hh]
            r = bwd_streams(sub(q), sub(k), sub(v), sub(g), sub(beta), S0[n, hh], sub(dO),
                            dS_T[n, hh], variant, chunk)
            dq[b, s:s + L][:, hh] = np.moveaxis(r[0], 0, 1)
            dk_[b, s:s + L][:, hh] = np.moveaxis(r[1], 0, 1)
            dvv[b, s:s + L][:, hh] = np.moveaxis(r[2], 0, 1)
            if dg is not None:
                dg[b, s:s + L][:, hh] = r[3].T
            if db is not None:
                db[b, s:s + L][:, hh] = r[4].T
            dS0[n, hh] = r[5]
    return dq, dk_, dvv, dg, db, dS0


def stream_work_flops(L: int, dk: int, dv: int) -> float:
    """Rough float64 flop count of fwd + bwd for one stream (for baseline reporting)."""
    return 29.0 * L * dk * dv


__all__ = ["VARIANTS", "fwd_streams", "bwd_streams", "oracle_fwd", "oracle_bwd",
           "stream_work_flops"]


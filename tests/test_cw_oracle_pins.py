"""Pins of the channel-wise float64 oracle (CPU only).

The general recurrence (paper Sec. 4.1, Eq. (gdn), per-channel g, b, w) is
checked against things other than its own loop:

* a brute-force unrolled recurrence with explicit d_k x d_k transition
  matrices (I - k (b*k)^T) Diag(e^g), for every chunk checkpoint and output;
* the scalar-gate oracle (pinned on its own): with g equal in every channel
  and b = w = beta (KDA with a scalar gate) every output and gradient equals
  it, dg and dbeta as channel sums; with b = 0, w = 1 it is the scalar-decay
  member;
* closed forms: LA (g = b = 0, w = 1) is causal linear attention; GLA
  (b = 0, w = 1) is masked attention with the per-channel decay e^{G_t - G_s}
  inside the score, and its final state has a closed form too; with b = 0 and
  w = 0 the state only decays;
* complex-step differentiation (Squire & Trapp 1998) of the forward for every
  gradient (full gates, GLA, KDA settings), central differences;
* packed sequences equal separate runs; planted mistakes in the forward and
  the backward fail the pins above.
"""
import numpy as np
import pytest

from oracle import cw_oracle as CW
from oracle import gdn_oracle as O


def _draw(seed, NS, L, dk, dv, *, decay=0.3, b_range=(0.0, 1.0), w_range=(0.0, 1.5), s0=0.3):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((NS, L, dk))
    k = rng.standard_normal((NS, L, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((NS, L, dv))
    g = -decay * np.log1p(np.exp(rng.standard_normal((NS, L, dk))))
    b = b_range[0] + (b_range[1] - b_range[0]) * rng.random((NS, L, dk))
    w = w_range[0] + (w_range[1] - w_range[0]) * rng.random((NS, L, dv))
    S0 = s0 * rng.standard_normal((NS, dk, dv))
    dO = rng.standard_normal((NS, L, dv))
    dST = rng.standard_normal((NS, dk, dv))
    return dict(q=q, k=k, v=v, g=g, b=b, w=w, S0=S0, dO=dO, dST=dST)


def rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def _dense_states(k, v, g, b, w, S0):
    """S_t for one stream from explicit transition matrices (all t, S_0 first)."""
    L, dk = k.shape
    S = S0.copy()
    out = [S.copy()]
    for t in range(L):
        kb = np.zeros(dk) if b is None else b[t] * k[t]
        wv = v[t] if w is None else w[t] * v[t]
        D = np.eye(dk) if g is None else np.diag(np.exp(g[t]))
        S = (np.eye(dk) - np.outer(k[t], kb)) @ D @ S + np.outer(k[t], wv)
        out.append(S.copy())
    return out


def _loss(o, ST, dO, dST):
    return (o * dO).sum(axis=(1, 2)) + (ST * dST).sum(axis=(1, 2))


# ---------------------------------------------------------------- forward pins

@pytest.mark.parametrize("gates", ["gbw", "g", "bw", "none", "b"])
def test_forward_matches_dense_transition_matrices(gates):
    L, dk, dv, chunk = 9, 4, 3, 4
    x = _draw(1, 1, L, dk, dv, b_range=(-0.3, 1.4))
    g = x["g"] if "g" in gates else None
    b = x["b"] if "b" in gates else None
    w = x["w"] if "w" in gates else None
    o, ST, st = CW.cw_fwd_streams(x["q"], x["k"], x["v"], g, b, w, x["S0"], chunk)
    Ss = _dense_states(x["k"][0], x["v"][0], None if g is None else g[0], None if b is None else b[0],
                       None if w is None else w[0], x["S0"][0])
    assert rel(ST[0], Ss[L]) < 1e-13
    for c in range(st.shape[1]):
        assert rel(st[0, c], Ss[c * chunk]) < 1e-13
    o_ref = np.stack([Ss[t + 1].T @ x["q"][0, t] for t in range(L)])
    assert rel(o[0], o_ref) < 1e-13


def test_scalar_gates_reduce_to_the_scalar_oracle():
    L, dk, dv, chunk = 11, 5, 4, 4
    x = _draw(2, 2, L, dk, dv)
    gs, beta = x["g"][:, :, 0], x["b"][:, :, 0]
    g = np.repeat(gs[:, :, None], dk, axis=2)
    b = np.repeat(beta[:, :, None], dk, axis=2)
    w = np.repeat(beta[:, :, None], dv, axis=2)
    a = CW.cw_fwd_streams(x["q"], x["k"], x["v"], g, b, w, x["S0"], chunk)
    r = O.fwd_streams(x["q"], x["k"], x["v"], gs, beta, x["S0"], "gated_delta", chunk)
    for u, vv in zip(a, r):
        assert rel(u, vv) < 1e-13
    ga = CW.cw_bwd_streams(x["q"], x["k"], x["v"], g, b, w, x["S0"], x["dO"], x["dST"], chunk)
    gr = O.bwd_streams(x["q"], x["k"], x["v"], gs, beta, x["S0"], x["dO"], x["dST"], "gated_delta", chunk)
    for i in (0, 1, 2):
        assert rel(ga[i], gr[i]) < 1e-12, i
    assert rel(ga[3].sum(-1), gr[3]) < 1e-12                      # dg: channel sum
    assert rel(ga[4].sum(-1) + ga[5].sum(-1), gr[4]) < 1e-12      # dbeta: erase + write gates
    assert rel(ga[6], gr[5]) < 1e-12


def test_no_erase_unit_write_is_the_scalar_decay_member():
    L, dk, dv, chunk = 10, 4, 3, 3
    x = _draw(3, 1, L, dk, dv)
    gs = x["g"][:, :, 0]
    g = np.repeat(gs[:, :, None], dk, axis=2)
    a = CW.cw_fwd_streams(x["q"], x["k"], x["v"], g, None, None, x["S0"], chunk)
    r = O.fwd_streams(x["q"], x["k"], x["v"], gs, None, x["S0"], "decay_only", chunk)
    for u, vv in zip(a, r):
        assert rel(u, vv) < 1e-13
    ga = CW.cw_bwd_streams(x["q"], x["k"], x["v"], g, None, None, x["S0"], x["dO"], x["dST"], chunk)
    gr = O.bwd_streams(x["q"], x["k"], x["v"], gs, None, x["S0"], x["dO"], x["dST"], "decay_only", chunk)
    for i in (0, 1, 2):
        assert rel(ga[i], gr[i]) < 1e-12
    assert rel(ga[3].sum(-1), gr[3]) < 1e-12
    assert ga[4] is None and ga[5] is None
    assert rel(ga[6], gr[5]) < 1e-12


def test_linear_attention_is_causal_attention_closed_form():
    L, dk, dv = 12, 5, 4
    x = _draw(4, 1, L, dk, dv)
    q, k, v, S0 = x["q"][0], x["k"][0], x["v"][0], x["S0"][0]
    o, ST, _ = CW.cw_fwd_streams(x["q"], x["k"], x["v"], None, None, None, x["S0"])
    scores = np.tril(q @ k.T)
    assert rel(o[0], q @ S0 + scores @ v) < 1e-13
    assert rel(ST[0], S0 + k.T @ v) < 1e-13


def test_gla_is_masked_attention_with_channel_decay():
    L, dk, dv = 12, 5, 4
    x = _draw(5, 1, L, dk, dv, decay=0.8)
    q, k, v, g, S0 = x["q"][0], x["k"][0], x["v"][0], x["g"][0], x["S0"][0]
    o, ST, _ = CW.cw_fwd_streams(x["q"], x["k"], x["v"], x["g"], None, None, x["S0"])
    G = np.cumsum(g, axis=0)                      # G_t = sum_{s <= t} g_s
    o_ref = np.zeros((L, dv))
    for t in range(L):
        o_ref[t] = (np.exp(G[t]) * q[t]) @ S0
        for s in range(t + 1):
            o_ref[t] += np.sum(q[t] * k[s] * np.exp(G[t] - G[s])) * v[s]
    assert rel(o[0], o_ref) < 1e-13
    ST_ref = np.exp(G[-1])[:, None] * S0 + sum(np.outer(np.exp(G[-1] - G[s]) * k[s], v[s]) for s in range(L))
    assert rel(ST[0], ST_ref) < 1e-13


def test_state_only_decays_without_erase_or_write():
    L, dk, dv = 7, 4, 3
    x = _draw(6, 1, L, dk, dv)
    w0 = np.zeros_like(x["w"])
    o, ST, _ = CW.cw_fwd_streams(x["q"], x["k"], x["v"], x["g"], None, w0, x["S0"])
    G = x["g"][0].sum(axis=0)
    assert rel(ST[0], np.exp(G)[:, None] * x["S0"][0]) < 1e-14
    # and without a decay either, the state is carried exactly
    o, ST, _ = CW.cw_fwd_streams(x["q"], x["k"], x["v"], None, None, w0, x["S0"])
    assert np.array_equal(ST[0], x["S0"][0])


# ---------------------------------------------------------------- backward pins

def _complex_step(x, g, b, w, chunk):
    """d loss / d input for every real input entry by complex-step differentiation."""
    h = 1e-30
    base = dict(q=x["q"], k=x["k"], v=x["v"], g=g, b=b, w=w, S0=x["S0"])
    out = {}
    for nm, arr in base.items():
        if arr is None:
            continue
        n = arr.size
        batch = {kk: (None if vv is None else np.repeat(vv.astype(np.complex128), n, axis=0))
                 for kk, vv in base.items()}
        pert = batch[nm].reshape(n, -1)
        pert[np.arange(n), np.arange(n)] += 1j * h
        o, ST, _ = CW.cw_fwd_streams(batch["q"], batch["k"], batch["v"], batch["g"], batch["b"],
                                     batch["w"], batch["S0"], chunk)
        Lc = _loss(o, ST, np.repeat(x["dO"], n, axis=0), np.repeat(x["dST"], n, axis=0))
        out[nm] = (Lc.imag / h).reshape(arr.shape)
    return out


@pytest.mark.parametrize("gates", ["gbw", "g", "gb", "bw", "none"])
def test_backward_matches_complex_step(gates):
    L, dk, dv, chunk = 7, 3, 4, 3  # chunks of 3, 3, 1 tokens
    x = _draw(7, 1, L, dk, dv, decay=0.5, b_range=(-0.4, 1.6))
    g = x["g"] if "g" in gates else None
    b = x["b"] if "b" in gates else None
    w = x["w"] if "w" in gates else None
    ref = _complex_step(x, g, b, w, chunk)
    r = CW.cw_bwd_streams(x["q"], x["k"], x["v"], g, b, w, x["S0"], x["dO"], x["dST"], chunk)
    got = dict(q=r[0], k=r[1], v=r[2], g=r[3], b=r[4], w=r[5], S0=r[6])
    got = {kk: vv for kk, vv in got.items() if vv is not None}
    assert set(got) == set(ref)
    for nm in ref:
        assert rel(got[nm], ref[nm]) < 1e-13, nm


def test_backward_matches_central_differences():
    L, dk, dv, chunk = 5, 3, 2, 2
    x = _draw(8, 1, L, dk, dv, decay=0.5)
    r = CW.cw_bwd_streams(x["q"], x["k"], x["v"], x["g"], x["b"], x["w"], x["S0"], x["dO"], x["dST"], chunk)
    got = dict(q=r[0], k=r[1], v=r[2], g=r[3], b=r[4], w=r[5], S0=r[6])
    base = {kk: x[kk] for kk in ("q", "k", "v", "g", "b", "w", "S0")}
    eps = 1e-6
    for nm, arr in base.items():
        fd = np.zeros_like(arr)
        for idx in np.ndindex(*arr.shape):
            vals = []
            for sgn in (1, -1):
                xx = arr.copy()
                xx[idx] += sgn * eps
                a = dict(base, **{nm: xx})
                o, ST, _ = CW.cw_fwd_streams(a["q"], a["k"], a["v"], a["g"], a["b"], a["w"], a["S0"], chunk)
                vals.append(_loss(o, ST, x["dO"], x["dST"])[0])
            fd[idx] = (vals[0] - vals[1]) / (2 * eps)
        assert rel(got[nm], fd) < 1e-7, nm


# ---------------------------------------------------------------- layout level

def test_packed_sequences_equal_separate_runs_bitwise():
    rng = np.random.default_rng(9)
    H, dk, dv = 2, 4, 3
    lens = [5, 1, 9]
    T = sum(lens)
    cu = np.concatenate([[0], np.cumsum(lens)])
    arr = lambda *s: rng.standard_normal(s)
    q, k, v = arr(1, T, H, dk), arr(1, T, H, dk), arr(1, T, H, dv)
    g, b, w = -0.3 * np.abs(arr(1, T, H, dk)), rng.random((1, T, H, dk)), rng.random((1, T, H, dv))
    S0, dO, dST = 0.3 * arr(3, H, dk, dv), arr(1, T, H, dv), arr(3, H, dk, dv)
    o, ST, st = CW.cw_oracle_fwd(q, k, v, g, b, w, S0, cu_seqlens=cu, chunk=4)
    grads = CW.cw_oracle_bwd(q, k, v, g, b, w, S0, dO, dST, cu_seqlens=cu, chunk=4)
    off = 0
    for n in range(3):
        s, L = cu[n], lens[n]
        sl = lambda t: t[:, s:s + L]
        o1, ST1, st1 = CW.cw_oracle_fwd(sl(q), sl(k), sl(v), sl(g), sl(b), sl(w), S0[n:n + 1], chunk=4)
        assert np.array_equal(o[:, s:s + L], o1) and np.array_equal(ST[n], ST1[0])
        nt = -(-L // 4)
        assert np.array_equal(st[off:off + nt], st1)
        off += nt
        g1 = CW.cw_oracle_bwd(sl(q), sl(k), sl(v), sl(g), sl(b), sl(w), S0[n:n + 1], sl(dO),
                              dST[n:n + 1], chunk=4)
        for a_, b_ in zip(grads[:6], g1[:6]):
            assert np.array_equal(a_[:, s:s + L], b_)
        assert np.array_equal(grads[6][n], g1[6][0])


def test_oracle_refuses_reduced_precision():
    x = _draw(10, 1, 3, 2, 2)
    with pytest.raises(TypeError):
        CW.cw_fwd_streams(x["q"].astype(np.float32), x["k"], x["v"], x["g"], x["b"], x["w"], x["S0"])


# -------------------------------------------------- pins have teeth (planted)

def test_planted_forward_mistake_is_caught(monkeypatch):
    """Erasing with the undecayed state (p = S^T (b*k) instead of St^T (b*k))
    fails the transition-matrix pin."""
    def broken(S, k_t, v_t, g_t, b_t, w_t):
        St = np.exp(g_t)[:, :, None] * S
        kb = b_t * k_t
        u = w_t * v_t - np.einsum("skv,sk->sv", S, kb)
        return St, kb, u, St + k_t[:, :, None] * u[:, None, :]

    x = _draw(11, 1, 6, 3, 2, decay=0.5)
    monkeypatch.setattr(CW, "_step", broken)
    _, ST, _ = CW.cw_fwd_streams(x["q"], x["k"], x["v"], x["g"], x["b"], x["w"], x["S0"])
    monkeypatch.undo()
    Ss = _dense_states(x["k"][0], x["v"][0], x["g"][0], x["b"][0], x["w"][0], x["S0"][0])
    assert rel(ST[0], Ss[6]) > 1e-3


def test_planted_backward_mistake_is_caught(monkeypatch):
    """Handing the post-update state where St is expected (a wrong dg and dkb
    contraction) fails the complex-step pin."""
    L, dk, dv, chunk = 5, 3, 3, 2
    x = _draw(12, 1, L, dk, dv, decay=0.5)
    ref = _complex_step(x, x["g"], x["b"], x["w"], chunk)
    real = CW._step

    def shifted(S, k_t, v_t, g_t, b_t, w_t):
        St, kb, u, Sn = real(S, k_t, v_t, g_t, b_t, w_t)
        return Sn, kb, u, Sn

    monkeypatch.setattr(CW, "_step", shifted)
    got = CW.cw_bwd_streams(x["q"], x["k"], x["v"], x["g"], x["b"], x["w"], x["S0"], x["dO"], x["dST"], chunk)
    monkeypatch.undo()
    assert rel(got[3][0], ref["g"]) > 1e-3

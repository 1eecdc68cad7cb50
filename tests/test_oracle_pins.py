"""Pins of the float64 oracle against things other than itself (CPU only).

* brute-force unrolled recurrence with explicit transition matrices (forward,
  every intermediate state, the chunk checkpoints);
* complex-step differentiation (Squire & Trapp 1998) of the oracle's own
  forward for every gradient, plus central finite differences;
* closed forms and invariants: beta = 0 and g = 0 give the identity map on the
  state (bitwise), beta = 0 gives S_T = exp(sum g) S0, the delta rule stores
  the value for a unit key with beta = 1, the scalar-decay member equals dense
  masked decayed attention, DeltaNet equals the gated rule at g = 0 (bitwise),
  the adjoint identity <dS0, X> = <dS_T, S_T(X) - S_T(0)>;
* the chunked reference equals the token-serial oracle (paper Sec. 4.1: paths
  that contract in different orders agree to 1e-12 in float64);
* packed sequences equal separate runs (bitwise).
"""
import numpy as np
import pytest

from oracle import chunked_ref as CR
from oracle import dense_ref as DR
from oracle import gdn_oracle as O


def _draw(seed, NS, L, dk, dv, *, unit_k=True, beta_range=(0, 1), decay=0.1, s0=0.3):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((NS, L, dk))
    k = rng.standard_normal((NS, L, dk))
    if unit_k:
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((NS, L, dv))
    lo, hi = beta_range
    beta = lo + (hi - lo) * rng.random((NS, L))
    g = -decay * np.log1p(np.exp(rng.standard_normal((NS, L))))
    S0 = s0 * rng.standard_normal((NS, dk, dv))
    dO = rng.standard_normal((NS, L, dv))
    dST = rng.standard_normal((NS, dk, dv))
    return q, k, v, g, beta, S0, dO, dST


def _gates(variant, g, beta):
    return (None if variant == "delta" else g), (None if variant == "decay_only" else beta)


def _bw(variant, beta, L):
    if variant == "decay_only":
        return np.zeros(L), np.ones(L)
    return beta, beta


def rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


# ---------------------------------------------------------------- forward pins

@pytest.mark.parametrize("variant", ["gated_delta", "delta", "decay_only"])
@pytest.mark.parametrize("unit_k", [True, False])
def test_forward_matches_unrolled_transition_matrices(variant, unit_k):
    L, dk, dv = 8, 4, 3
    q, k, v, g, beta, S0, _, _ = _draw(1, 1, L, dk, dv, unit_k=unit_k, beta_range=(-0.5, 1.7))
    gg, bb = _gates(variant, g, beta)
    o, ST, states = O.fwd_streams(q, k, v, gg, bb, S0, variant, chunk=3)
    g0 = np.zeros(L) if variant == "delta" else g[0]
    b, w = _bw(variant, beta[0], L)
    Ss = DR.unrolled_states(k[0], v[0], g0, b, w, S0[0])
    for t in range(L):
        assert rel(o[0, t], Ss[t + 1].T @ q[0, t]) < 1e-13
    assert rel(ST[0], Ss[L]) < 1e-13
    # chunk checkpoints: the state before tokens 0, 3, 6
    for c in range(3):
        assert rel(states[0, c], Ss[3 * c]) < 1e-13 or np.all(states[0, c] == Ss[3 * c])


def test_scalar_decay_member_is_dense_masked_attention():
    L, dk, dv = 40, 5, 4
    q, k, v, g, _, S0, _, _ = _draw(2, 1, L, dk, dv, decay=1.0)
    o, ST, _ = O.fwd_streams(q, k, v, g, None, S0, "decay_only", chunk=16)
    Od, STd = DR.decay_attention(q[0], k[0], v[0], g[0], S0[0])
    assert rel(o[0], Od) < 1e-12
    assert rel(ST[0], STd) < 1e-12


def test_identity_state_when_beta_and_g_vanish():
    L, dk, dv = 70, 6, 5
    q, k, v, g, beta, S0, _, _ = _draw(3, 2, L, dk, dv)
    o, ST, states = O.fwd_streams(q, k, v, np.zeros_like(g), np.zeros_like(beta), S0,
                                  "gated_delta", chunk=64)
    assert np.array_equal(ST, S0)
    assert np.array_equal(states[:, 1], S0)
    ref = np.einsum("skv,stk->stv", S0, q)
    assert rel(o, ref) < 1e-15


def test_beta_zero_gives_pure_decay_closed_form():
    L, dk, dv = 50, 4, 4
    q, k, v, g, beta, S0, _, _ = _draw(4, 2, L, dk, dv)
    _, ST, _ = O.fwd_streams(q, k, v, g, np.zeros_like(beta), S0, "gated_delta")
    expect = np.exp(g.sum(axis=1))[:, None, None] * S0
    assert rel(ST, expect) < 1e-14


def test_delta_rule_stores_the_value_for_unit_keys():
    L, dk, dv = 12, 5, 3
    rng = np.random.default_rng(5)
    q, _, v, g, _, S0, _, _ = _draw(5, 1, L, dk, dv)
    idx = rng.integers(0, dk, size=L)
    sgn = rng.choice([-1.0, 1.0], size=L)
    k = np.zeros((1, L, dk))
    k[0, np.arange(L), idx] = sgn
    beta = np.ones((1, L))
    # run one token at a time to read S_t after each token
    S = S0.copy()
    for t in range(L):
        _, S, _ = O.fwd_streams(q[:, t:t + 1], k[:, t:t + 1], v[:, t:t + 1], g[:, t:t + 1],
                                beta[:, t:t + 1], S, "gated_delta")
        assert rel(S[0].T @ k[0, t], v[0, t]) < 1e-14


def test_deltanet_equals_gated_rule_at_zero_decay_bitwise():
    L, dk, dv = 33, 4, 6
    q, k, v, g, beta, S0, dO, dST = _draw(6, 2, L, dk, dv)
    a = O.fwd_streams(q, k, v, None, beta, S0, "delta", chunk=8)
    b = O.fwd_streams(q, k, v, np.zeros_like(g), beta, S0, "gated_delta", chunk=8)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    ga = O.bwd_streams(q, k, v, None, beta, S0, dO, dST, "delta", chunk=8)
    gb = O.bwd_streams(q, k, v, np.zeros_like(g), beta, S0, dO, dST, "gated_delta", chunk=8)
    for i in (0, 1, 2, 4, 5):
        assert np.array_equal(ga[i], gb[i])


# --------------------------------------------------------------- backward pins

def _loss(o, ST, dO, dST):
    return np.sum(dO * o, axis=(1, 2)) + np.sum(dST * ST, axis=(1, 2))


def _complex_step_grads(variant, q, k, v, g, beta, S0, dO, dST, chunk):
    """d loss / d input for every entry, one perturbed copy of the stream per entry."""
    h = 1e-30
    names = ["q", "k", "v", "g", "beta", "S0"]
    base = dict(q=q, k=k, v=v, g=g, beta=beta, S0=S0)
    out = {}
    for nm in names:
        if base[nm] is None:
            continue
        x = base[nm][0]
        n = x.size
        batch = {key: (None if val is None else np.repeat(val.astype(np.complex128), n, axis=0))
                 for key, val in base.items()}
        pert = batch[nm].reshape(n, -1)
        pert[np.arange(n), np.arange(n)] += 1j * h
        o, ST, _ = O.fwd_streams(batch["q"], batch["k"], batch["v"], batch["g"], batch["beta"],
                                 batch["S0"], variant, chunk)
        Lc = _loss(o, ST, np.repeat(dO, n, axis=0), np.repeat(dST, n, axis=0))
        out[nm] = (Lc.imag / h).reshape(x.shape)
    return out


@pytest.mark.parametrize("variant", ["gated_delta", "delta", "decay_only"])
@pytest.mark.parametrize("unit_k,beta_range", [(True, (0, 1)), (False, (-0.4, 1.6))])
def test_backward_matches_complex_step(variant, unit_k, beta_range):
    L, dk, dv, chunk = 7, 3, 4, 3  # chunks of 3, 3, 1 tokens
    q, k, v, g, beta, S0, dO, dST = _draw(7, 1, L, dk, dv, unit_k=unit_k, beta_range=beta_range,
                                          decay=0.5)
    gg, bb = _gates(variant, g, beta)
    ref = _complex_step_grads(variant, q, k, v, gg, bb, S0, dO, dST, chunk)
    dq, dk_, dv_, dg, db, dS0 = O.bwd_streams(q, k, v, gg, bb, S0, dO, dST, variant, chunk)
    got = dict(q=dq[0], k=dk_[0], v=dv_[0], S0=dS0[0])
    if dg is not None:
        got["g"] = dg[0]
    if db is not None:
        got["beta"] = db[0]
    assert set(got) == set(ref)
    for nm in ref:
        assert rel(got[nm], ref[nm]) < 1e-13, nm


def test_backward_matches_central_differences():
    L, dk, dv, chunk = 6, 3, 2, 4
    q, k, v, g, beta, S0, dO, dST = _draw(8, 1, L, dk, dv, decay=0.5)
    dq, dk_, dv_, dg, db, dS0 = O.bwd_streams(q, k, v, g, beta, S0, dO, dST, "gated_delta", chunk)
    base = dict(q=q, k=k, v=v, g=g, beta=beta, S0=S0)
    got = dict(q=dq, k=dk_, v=dv_, g=dg, beta=db, S0=dS0)
    eps = 1e-6
    for nm, x in base.items():
        fd = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args_p = dict(base, **{nm: xp})
            args_m = dict(base, **{nm: xm})
            op, STp, _ = O.fwd_streams(**args_p, variant="gated_delta", chunk=chunk)
            om, STm, _ = O.fwd_streams(**args_m, variant="gated_delta", chunk=chunk)
            fd[idx] = (_loss(op, STp, dO, dST) - _loss(om, STm, dO, dST))[0] / (2 * eps)
        assert rel(got[nm], fd) < 1e-7, nm


def test_adjoint_identity_for_initial_state():
    L, dk, dv = 20, 4, 3
    q, k, v, g, beta, S0, _, dST = _draw(9, 1, L, dk, dv)
    X = np.random.default_rng(10).standard_normal(S0.shape)
    zeros_dO = np.zeros((1, L, dv))
    dS0 = O.bwd_streams(q, k, v, g, beta, X, zeros_dO, dST, "gated_delta")[5]
    _, ST_X, _ = O.fwd_streams(q, k, v, g, beta, X, "gated_delta")
    _, ST_0, _ = O.fwd_streams(q, k, v, g, beta, np.zeros_like(X), "gated_delta")
    lhs = np.sum(dS0 * X)
    rhs = np.sum(dST * (ST_X - ST_0))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(rhs))


# -------------------------------------------------- chunked = sequential (I4)

@pytest.mark.parametrize("variant", ["gated_delta", "delta", "decay_only"])
@pytest.mark.parametrize("C", [1, 3, 16, 64])
@pytest.mark.parametrize("L", [1, 63, 64, 65, 200])
def test_chunked_reference_equals_token_serial(variant, C, L):
    dk, dv = 6, 5
    q, k, v, g, beta, S0, dO, dST = _draw(11 + L, 1, L, dk, dv, decay=0.3)
    gg, bb = _gates(variant, g, beta)
    o, ST, st = O.fwd_streams(q, k, v, gg, bb, S0, variant, chunk=C)
    f = CR.chunked_fwd(q[0], k[0], v[0], None if gg is None else gg[0],
                       None if bb is None else bb[0], S0[0], variant, C)
    assert rel(f[0], o[0]) < 1e-12 and rel(f[1], ST[0]) < 1e-12 and rel(f[2], st[0]) < 1e-12
    r = O.bwd_streams(q, k, v, gg, bb, S0, dO, dST, variant, chunk=64)
    b = CR.chunked_bwd(q[0], k[0], v[0], None if gg is None else gg[0],
                       None if bb is None else bb[0], S0[0], dO[0], dST[0], variant, C)
    for i in range(6):
        if r[i] is None:
            assert b[i] is None
            continue
        assert rel(b[i], r[i][0]) < 1e-12, i


def test_scalar_decay_member_has_identity_inverse_bitwise():
    L, dk, dv = 100, 4, 4
    q, k, v, g, _, S0, _, _ = _draw(12, 1, L, dk, dv)
    *_, inter = CR.chunked_fwd(q[0], k[0], v[0], g[0], None, S0[0], "decay_only", 64, keep=True)
    for st in inter:
        n = st["T"].shape[0]
        assert np.array_equal(st["T"], np.eye(n))
        assert np.array_equal(st["W"], np.zeros_like(st["W"]))


def test_forward_substitution_is_an_inverse():
    rng = np.random.default_rng(13)
    A = np.tril(rng.standard_normal((20, 20)), -1) * 0.3
    T = CR.forward_substitution_inverse(A)
    assert np.abs(T @ (np.eye(20) + A) - np.eye(20)).max() < 1e-12
    assert np.array_equal(np.triu(T, 1), np.zeros_like(T))
    assert np.array_equal(np.diag(T), np.ones(20))


# ------------------------------------------------------------ layout / varlen

def test_packed_sequences_equal_separate_runs_bitwise():
    rng = np.random.default_rng(14)
    H, dk, dv = 2, 4, 3
    lens = [5, 70, 1, 64, 0, 130]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    N = len(lens)
    q = rng.standard_normal((1, T, H, dk))
    k = rng.standard_normal((1, T, H, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((1, T, H, dv))
    g = -0.1 * rng.random((1, T, H))
    beta = rng.random((1, T, H))
    S0 = rng.standard_normal((N, H, dk, dv))
    dO = rng.standard_normal((1, T, H, dv))
    dST = rng.standard_normal((N, H, dk, dv))
    o, ST, st = O.oracle_fwd(q, k, v, g, beta, S0, cu_seqlens=cu)
    grads = O.oracle_bwd(q, k, v, g, beta, S0, dO, dST, cu_seqlens=cu)
    off = 0
    for n, L in enumerate(lens):
        s = int(cu[n])
        sl = slice(s, s + L)
        o1, ST1, st1 = O.oracle_fwd(q[:, sl], k[:, sl], v[:, sl], g[:, sl], beta[:, sl], S0[n:n + 1])
        assert np.array_equal(o[:, sl], o1) and np.array_equal(ST[n], ST1[0])
        nt = -(-L // 64)
        assert np.array_equal(st[off:off + nt], st1)
        off += nt
        g1 = O.oracle_bwd(q[:, sl], k[:, sl], v[:, sl], g[:, sl], beta[:, sl], S0[n:n + 1],
                          dO[:, sl], dST[n:n + 1])
        for i in range(5):
            assert np.array_equal(grads[i][:, sl], g1[i])
        assert np.array_equal(grads[5][n], g1[5][0])
    assert off == st.shape[0]


def test_empty_sequence_returns_initial_state():
    q = np.zeros((1, 0, 1, 4))
    v = np.zeros((1, 0, 1, 3))
    g = np.zeros((1, 0, 1))
    S0 = np.random.default_rng(15).standard_normal((1, 1, 4, 3))
    dST = np.random.default_rng(16).standard_normal((1, 1, 4, 3))
    o, ST, st = O.oracle_fwd(q, q, v, g, g, S0)
    assert o.shape == (1, 0, 1, 3) and st.shape == (0, 1, 4, 3) and np.array_equal(ST, S0)
    r = O.oracle_bwd(q, q, v, g, g, S0, v, dST)
    assert np.array_equal(r[5], dST)


def test_oracle_refuses_reduced_precision():
    x = np.zeros((1, 2, 3), np.float32)
    with pytest.raises(TypeError):
        O.fwd_streams(x, x, x, np.zeros((1, 2), np.float32), np.zeros((1, 2), np.float32),
                      np.zeros((1, 3, 3), np.float32))
    with pytest.raises(TypeError):
        CR.chunked_fwd(x[0], x[0], x[0], None, np.zeros(2, np.float32), np.zeros((3, 3)), "delta")


# ---------------------------------------------------- non-finite class contract

def test_nonfinite_classes_follow_the_formula_order():
    """NaN in one v row and +Inf in one g entry: the classes the loop fixes."""
    L, dk, dv = 40, 4, 3
    q, k, v, g, beta, S0, dO, dST = _draw(17, 1, L, dk, dv)
    t_nan, t_inf = 30, 12
    v[0, t_nan] = np.nan
    g[0, t_inf] = np.inf
    o, ST, _ = O.fwd_streams(q, k, v, g, beta, S0, "gated_delta", chunk=16)
    assert np.all(np.isfinite(o[0, :t_inf]))
    assert not np.any(np.isfinite(o[0, t_inf:]))
    dq, dk_, dv_, dg, db, dS0 = O.bwd_streams(q, k, v, g, beta, S0, dO, dST, "gated_delta", 16)
    # dq before the Inf decay only reads the forward state, which is finite there
    assert np.all(np.isfinite(dq[0, :t_inf]))
    # everything propagated backward through exp(+Inf) * dSt is NaN before t_inf
    assert np.all(np.isnan(dk_[0, :t_inf])) and np.all(np.isnan(dv_[0, :t_inf]))
    assert np.all(np.isnan(dg[0, :t_inf])) and np.all(np.isnan(db[0, :t_inf]))
    assert np.all(np.isnan(dS0))


# -------------------------------------------------- pins have teeth (planted)

def test_planted_forward_mistake_is_caught(monkeypatch):
    """Dropping beta from the write makes the unrolled-matrix pin fail."""
    real = O._step_fwd

    def broken(S, k_t, v_t, g_t, b_t, variant):
        St = np.exp(g_t)[:, None, None] * S
        p = np.einsum("skv,sk->sv", St, k_t)
        u = v_t - b_t[:, None] * p  # wrong grouping: beta * (v - p) expected
        return St, p, u, St + k_t[:, :, None] * u[:, None, :]

    monkeypatch.setattr(O, "_step_fwd", broken)
    L, dk, dv = 6, 3, 2
    q, k, v, g, beta, S0, _, _ = _draw(18, 1, L, dk, dv)
    _, ST, _ = O.fwd_streams(q, k, v, g, beta, S0, "gated_delta")
    Ss = DR.unrolled_states(k[0], v[0], g[0], beta[0], beta[0], S0[0])
    assert rel(ST[0], Ss[L]) > 1e-3
    monkeypatch.setattr(O, "_step_fwd", real)


def test_planted_backward_mistake_is_caught(monkeypatch):
    """A transposed dg contraction (<dSt, S_t> instead of <dSt, St>) fails complex step."""
    L, dk, dv, chunk = 5, 3, 3, 2
    q, k, v, g, beta, S0, dO, dST = _draw(19, 1, L, dk, dv, decay=0.5)
    ref = _complex_step_grads("gated_delta", q, k, v, g, beta, S0, dO, dST, chunk)
    real_step = O._step_fwd

    def shifted(S, k_t, v_t, g_t, b_t, variant):
        St, p, u, Sn = real_step(S, k_t, v_t, g_t, b_t, variant)
        return Sn, p, u, Sn  # hands the post-update state where St is expected

    monkeypatch.setattr(O, "_step_fwd", shifted)
    got = O.bwd_streams(q, k, v, g, beta, S0, dO, dST, "gated_delta", chunk)
    monkeypatch.setattr(O, "_step_fwd", real_step)
    assert rel(got[3][0], ref["g"]) > 1e-3

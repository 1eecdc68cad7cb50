"""Pins of the oracle's layout entry points (CPU only).

``oracle_fwd`` / ``oracle_bwd`` and ``cw_oracle_fwd`` / ``cw_oracle_bwd`` gather
each (sequence, head) stream out of the API layout ([B,T,H,d] token-major, gates
[B,T,H] or [B,T,H,d], states [N,H,dk,dv], chunk states [sum_n NT_n, H, dk, dv]),
run the stream-batched cores on it and scatter the results back.  Every GPU
parity test goes through that gather/scatter, so it is pinned here against an
independent one: each stream is cut out with plain indexing ``x[b, s:s+L, h]``,
run alone through ``fwd_streams`` / ``bwd_streams`` (``cw_*_streams``), and
every entry of the layout-level result must equal it bitwise.  Entries of heads
outside ``heads=`` must stay NaN.  Shapes use B >= 2, H >= 3, packed sequences
with an empty one and ragged chunk tails, and unsorted head subsets.  Planted
mistakes in the oracle's gather or scatter (two heads swapped, a chunk offset
off by one) must be caught.
"""
import numpy as np
import pytest

import workloads as W
from oracle import cw_oracle as CW
from oracle import gdn_oracle as O

CH = 16  # a small chunk keeps several chunk states per stream at small T


def _f64(x):
    return None if x is None else x.astype(np.float64)


def _streams(B, T, cu):
    """(batch row, first token, length) of every sequence, written out directly."""
    if cu is None:
        return [(b, 0, T) for b in range(B)]
    return [(0, int(cu[n]), int(cu[n + 1]) - int(cu[n])) for n in range(len(cu) - 1)]


def _one(x, b, s, L, h):
    """Stream (b, h) of an API-layout tensor as a batch of one stream."""
    return None if x is None else np.ascontiguousarray(x[b, s:s + L, h])[None]


def _expected_fwd(core, acts, gates, S0, B, T, H, cu, heads, chunk):
    """Forward results assembled stream by stream from the core (reference scatter)."""
    q = acts[0]
    dv = acts[2].shape[-1]
    dk = q.shape[-1]
    seqs = _streams(B, T, cu)
    nts = [-(-L // chunk) for (_, _, L) in seqs]
    o = np.full((B, T, H, dv), np.nan)
    S_T = np.full((len(seqs), H, dk, dv), np.nan)
    st = np.full((sum(nts), H, dk, dv), np.nan)
    first = 0
    for n, (b, s, L) in enumerate(seqs):
        for h in heads:
            args = [_one(x, b, s, L, h) for x in acts] + [_one(x, b, s, L, h) for x in gates]
            o1, ST1, st1 = core(*args, S0[n, h][None], chunk=chunk)
            for t in range(L):
                o[b, s + t, h] = o1[0, t]
            S_T[n, h] = ST1[0]
            for c in range(nts[n]):
                st[first + c, h] = st1[0, c]
        first += nts[n]
    return o, S_T, st


def _expected_bwd(core, acts, gates, S0, dO, dST, B, T, H, cu, heads, chunk):
    """Backward results assembled stream by stream: activation gradients, gate
    gradients (same layout as their gate), dS0."""
    seqs = _streams(B, T, cu)
    grads_act = [np.full(x.shape, np.nan) for x in acts]
    grads_gate = [None if x is None else np.full(x.shape, np.nan) for x in gates]
    dS0 = np.full(S0.shape, np.nan)
    for n, (b, s, L) in enumerate(seqs):
        for h in heads:
            args = [_one(x, b, s, L, h) for x in acts] + [_one(x, b, s, L, h) for x in gates]
            r = core(*args, S0[n, h][None], _one(dO, b, s, L, h), dST[n, h][None], chunk=chunk)
            na = len(acts)
            for i in range(na):
                for t in range(L):
                    grads_act[i][b, s + t, h] = r[i][0, t]
            for i, gg in enumerate(grads_gate):
                if gg is not None:
                    for t in range(L):
                        gg[b, s + t, h] = r[na + i][0, t]
            dS0[n, h] = r[-1][0]
    return grads_act, grads_gate, dS0


def _same(a, b):
    """Bitwise equality, NaN in the same places counting as equal."""
    return a.shape == b.shape and np.array_equal(a, b, equal_nan=True)


# ---------------------------------------------------------------- scalar gates

def _scalar_case(variant, packed, B=2, H=3, seed=3):
    if packed:
        cu = np.array([0, 21, 21, 54, 70], np.int32)  # an empty sequence, ragged tails
        c = W.make_case("layout", B=1, T=int(cu[-1]), H=H, dk=8, dv=6, io_dtype="f32",
                        variant=variant, cu_seqlens=cu, seed=seed, decay_scale=0.3)
    else:
        c = W.make_case("layout", B=B, T=37, H=H, dk=8, dv=6, io_dtype="f32", variant=variant,
                        seed=seed, decay_scale=0.3)
    return c


def _scalar_check(c, heads, fwd=O.oracle_fwd, bwd=O.oracle_bwd):
    """List of mismatching outputs between the layout entry points and the per-stream reference."""
    q, k, v, dO = (_f64(x) for x in (c.q, c.k, c.v, c.dO))
    g, b = _f64(c.g), _f64(c.beta)
    S0, dST = _f64(c.S0), _f64(c.dS_T)
    hs = list(range(c.H)) if heads is None else list(heads)

    def core_f(q1, k1, v1, g1, b1, S01, chunk):
        return O.fwd_streams(q1, k1, v1, g1, b1, S01, c.variant, chunk)

    def core_b(q1, k1, v1, g1, b1, S01, dO1, dST1, chunk):
        return O.bwd_streams(q1, k1, v1, g1, b1, S01, dO1, dST1, c.variant, chunk)

    bad = []
    got = fwd(q, k, v, g, b, S0, variant=c.variant, cu_seqlens=c.cu_seqlens, chunk=CH, heads=heads)
    exp = _expected_fwd(core_f, [q, k, v], [g, b], S0, c.B, c.T, c.H, c.cu_seqlens, hs, CH)
    for nm, x, y in zip(("o", "S_T", "states"), got, exp):
        if not _same(x, y):
            bad.append(nm)
    got = bwd(q, k, v, g, b, S0, dO, dST, variant=c.variant, cu_seqlens=c.cu_seqlens, chunk=CH,
              heads=heads)
    ea, eg, eS0 = _expected_bwd(core_b, [q, k, v], [g, b], S0, dO, dST, c.B, c.T, c.H,
                                c.cu_seqlens, hs, CH)
    for nm, x, y in zip(("dq", "dk", "dv", "dg", "dbeta", "dS0"), got, ea + eg + [eS0]):
        if (x is None) != (y is None) or (x is not None and not _same(x, y)):
            bad.append(nm)
    return bad


@pytest.mark.parametrize("variant", ["gated_delta", "delta", "decay_only"])
@pytest.mark.parametrize("packed", [False, True])
@pytest.mark.parametrize("heads", [None, [2, 0], [1]])
def test_scalar_layout_matches_streams(variant, packed, heads):
    c = _scalar_case(variant, packed)
    assert _scalar_check(c, heads) == []


def test_scalar_layout_subset_leaves_other_heads_nan():
    c = _scalar_case("gated_delta", False)
    o, S_T, st = O.oracle_fwd(*(_f64(x) for x in (c.q, c.k, c.v, c.g, c.beta, c.S0)), chunk=CH,
                              heads=[2, 0])
    assert np.isnan(o[:, :, 1]).all() and np.isnan(S_T[:, 1]).all() and np.isnan(st[:, 1]).all()
    assert np.isfinite(o[:, :, [0, 2]]).all() and np.isfinite(st[:, [0, 2]]).all()


def test_scalar_layout_batch_rows_differ():
    # B = 2 with distinct inputs per row: a gather that ignored the batch index
    # would give equal rows
    c = _scalar_case("gated_delta", False)
    o, _, _ = O.oracle_fwd(*(_f64(x) for x in (c.q, c.k, c.v, c.g, c.beta, c.S0)), chunk=CH)
    assert not np.allclose(o[0], o[1])


def _swap_heads_gather(orig, h1=0, h2=1):
    def gather(x, b, s, L):
        y = orig(x, b, s, L)
        if y is None:
            return None
        y = y.copy()
        y[[h1, h2]] = y[[h2, h1]]
        return y
    return gather


@pytest.mark.parametrize("packed", [False, True])
def test_scalar_layout_planted_head_swap_is_caught(monkeypatch, packed):
    c = _scalar_case("gated_delta", packed)
    monkeypatch.setattr(O, "_gather", _swap_heads_gather(O._gather))
    assert {"o", "states", "dq", "dk", "dv", "dg", "dbeta"} <= set(_scalar_check(c, None))


def test_scalar_layout_planted_chunk_offset_is_caught():
    # a scatter that puts sequence n's chunk states one entry too far
    c = _scalar_case("gated_delta", True)

    def fwd_shifted(*a, **kw):
        o, S_T, st = O.oracle_fwd(*a, **kw)
        st2 = np.full_like(st, np.nan)
        st2[1:] = st[:-1]
        return o, S_T, st2

    assert "states" in _scalar_check(c, None, fwd=fwd_shifted)


# ---------------------------------------------------------------- channel-wise gates

def _cw_case(gates, packed, seed=5):
    if packed:
        cu = np.array([0, 19, 19, 51, 66], np.int32)
        return W.make_cw_case("cw_layout", 1, int(cu[-1]), 3, 8, 6, gates=gates, seed=seed, cu_seqlens=cu)
    return W.make_cw_case("cw_layout", 2, 35, 3, 8, 6, gates=gates, seed=seed)


def _cw_check(c, heads, fwd=CW.cw_oracle_fwd, bwd=CW.cw_oracle_bwd):
    q, k, v, dO = (_f64(x) for x in (c.q, c.k, c.v, c.dO))
    g, b, w = _f64(c.g), _f64(c.b), _f64(c.w)
    S0, dST = _f64(c.S0), _f64(c.dS_T)
    hs = list(range(c.H)) if heads is None else list(heads)
    bad = []
    got = fwd(q, k, v, g, b, w, S0, cu_seqlens=c.cu_seqlens, chunk=CH, heads=heads)
    exp = _expected_fwd(CW.cw_fwd_streams, [q, k, v], [g, b, w], S0, c.B, c.T, c.H, c.cu_seqlens, hs, CH)
    for nm, x, y in zip(("o", "S_T", "states"), got, exp):
        if not _same(x, y):
            bad.append(nm)
    got = bwd(q, k, v, g, b, w, S0, dO, dST, cu_seqlens=c.cu_seqlens, chunk=CH, heads=heads)
    ea, eg, eS0 = _expected_bwd(CW.cw_bwd_streams, [q, k, v], [g, b, w], S0, dO, dST, c.B, c.T, c.H,
                                c.cu_seqlens, hs, CH)
    for nm, x, y in zip(("dq", "dk", "dv", "dg", "db", "dw", "dS0"), got, ea + eg + [eS0]):
        if (x is None) != (y is None) or (x is not None and not _same(x, y)):
            bad.append(nm)
    return bad


@pytest.mark.parametrize("gates", ["gbw", "kda", "g", ""])
@pytest.mark.parametrize("packed", [False, True])
@pytest.mark.parametrize("heads", [None, [2, 0]])
def test_cw_layout_matches_streams(gates, packed, heads):
    assert _cw_check(_cw_case(gates, packed), heads) == []


@pytest.mark.parametrize("packed", [False, True])
def test_cw_layout_planted_head_swap_is_caught(monkeypatch, packed):
    c = _cw_case("gbw", packed)
    monkeypatch.setattr(CW, "_gather", _swap_heads_gather(CW._gather))
    assert {"o", "states", "dq", "dk", "dv", "dg", "db", "dw"} <= set(_cw_check(c, None))

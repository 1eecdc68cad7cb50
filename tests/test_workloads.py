"""The seeded input generator: determinism, rounding and the varlen recipe (CPU)."""
import numpy as np
import torch

import workloads as W


def test_same_seed_same_bits():
    a = W.make_case("a", B=1, T=70, H=2, dk=8, dv=16)
    b = W.make_case("b", B=1, T=70, H=2, dk=8, dv=16)
    for x, y in ((a.q, b.q), (a.v, b.v), (a.g, b.g), (a.beta, b.beta), (a.S0, b.S0), (a.dO, b.dO)):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    x[:4] = [np.inf, -np.inf, 0.0, -0.0]
    ours = W.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))
    assert np.isnan(W.round_bf16(np.array([np.nan], np.float32)))[0]


def test_activations_are_bf16_representable_and_gates_in_range():
    c = W.make_case("c", B=2, T=33, H=3, dk=16, dv=8)
    for x in (c.q, c.k, c.v, c.dO):
        assert np.array_equal(W.round_bf16(x), x)
    assert np.all((c.beta > 0) & (c.beta < 1))
    assert np.all(c.g <= 0)
    nq = np.linalg.norm(c.q.astype(np.float64), axis=-1)
    assert np.all(np.abs(nq - 1) < 1e-2)


def test_varlen_recipe_hits_total_and_bounds():
    cu = W.config4_cu_seqlens()
    L = np.diff(cu)
    assert cu[0] == 0 and cu[-1] == 32768 and len(L) == 16
    assert np.all((L >= 64) & (L <= 4096))


def test_zero_std_gives_positive_zero_and_keeps_draw_order():
    a = W.make_case("a", B=1, T=10, H=1, dk=4, dv=4, S0_std=0.0, dST_std=0.0)
    b = W.make_case("b", B=1, T=10, H=1, dk=4, dv=4)
    assert np.array_equal(a.S0.view(np.uint32), np.zeros_like(a.S0.view(np.uint32)))
    assert np.array_equal(a.dO, b.dO)


def test_injection_positions_and_variants():
    c = W.make_case("n", B=2, T=50, H=2, dk=4, dv=4, inject="row")
    b1, t1, h1, _ = c.injected["v_nan"]
    assert np.all(np.isnan(c.v[b1, t1, h1]))
    b2, t2, h2 = c.injected["g_inf"]
    assert c.g[b2, t2, h2] == np.inf
    assert np.isfinite(c.q).all() and np.isfinite(c.k).all()
    d = W.make_case("d", B=1, T=5, H=1, dk=4, dv=4, variant="delta")
    assert d.g is None and d.beta is not None
    e = W.make_case("e", B=1, T=5, H=1, dk=4, dv=4, variant="decay_only")
    assert e.beta is None and e.g is not None

"""Tolerance-free NaN/Inf semantics of the scalar-gate path, input by input.

A stream whose inputs hold a NaN or an Inf is recomputed token by token in the
oracle's operation order, so every output element must have the oracle's class
(finite, NaN, +Inf, -Inf) exactly; finite entries must still meet the rel-L2
bar.  Each case poisons one input: an element of q, k, v or dO, one gate entry
of g or beta (g = +Inf, or -Inf: an exact reset of the state that leaves every
output finite), or one element of S0 or dS_T, for both I/O
dtypes, all three family members and every instantiated value width, so each
kernel's non-finite flag and the routing to the exact pass are exercised
(including the exact backward at d_k = 128).  Clean streams of the same call
must stay finite.
"""
import zlib

import numpy as np
import pytest

import workloads as W
from tests import harness as Hn

pytestmark = pytest.mark.gpu

POISON = {"q": np.inf, "k": np.nan, "v": np.nan, "dO": -np.inf, "g": np.inf, "g_neg": -np.inf,
          "beta": np.nan, "S0": np.nan, "dS_T": np.inf}


def _applies(inp, variant):
    if inp in ("g", "g_neg"):
        return variant != "delta"
    if inp == "beta":
        return variant != "decay_only"
    return True


def _poison(case, inp, seed):
    """One poisoned entry (position from a generator seeded per case); returns (b or n, h)."""
    rng = np.random.default_rng(seed)
    val = np.float32(POISON[inp])
    if inp in ("S0", "dS_T"):
        x = getattr(case, inp)
        n, h = int(rng.integers(x.shape[0])), int(rng.integers(case.H))
        x[n, h, int(rng.integers(case.dk)), int(rng.integers(case.dv))] = val
        return n, h
    name = "g" if inp == "g_neg" else inp
    x = getattr(case, name)
    b, h = int(rng.integers(case.B)), int(rng.integers(case.H))
    t = int(rng.integers(case.T // 4, case.T))
    if x.ndim == 4:
        x[b, t, h, int(rng.integers(x.shape[-1]))] = val
    else:
        x[b, t, h] = val
    return b, h


def _run(case, inp, seed):
    b, h = _poison(case, inp, seed)
    print("case", W.describe(case), "poison", inp, "stream", (b, h), flush=True)
    dev, ref = Hn.run_device(case), Hn.run_oracle(case)
    res = Hn.compare(dev, ref)
    print({k: (f"{v[0]:.2e}", v[1]) for k, v in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL[case.io_dtype], f"{case.name} {inp}")
    # the poison reached some output, and only its own stream.  g = -Inf is the
    # exception: exp(-Inf) = 0 erases the state exactly, every term of the
    # recurrence and of its adjoint stays finite (dg_t = <dSt, St> = 0), and the
    # outputs must stay finite too
    poisoned = any(not np.isfinite(x).all() for x in ref.values() if x is not None)
    assert poisoned == (inp != "g_neg"), (inp, poisoned)
    if inp == "g_neg":
        assert all(np.isfinite(x).all() for x in dev.values() if x is not None)
    for nm in ("o", "dq", "dk", "dv"):
        x = dev[nm]
        for bb in range(case.B):
            for hh in range(case.H):
                if (bb, hh) != (b, h):
                    assert np.isfinite(x[bb, :, hh]).all(), (nm, bb, hh)


@pytest.mark.parametrize("inp", list(POISON))
@pytest.mark.parametrize("dv", [64, 256])
@pytest.mark.parametrize("variant", ["gated_delta", "delta", "decay_only"])
@pytest.mark.parametrize("io", ["bf16", "f32"])
def test_poisoned_input(io, variant, dv, inp):
    if not _applies(inp, variant):
        pytest.skip(f"{variant} has no {inp}")
    seed = zlib.crc32(f"{io}/{variant}/{dv}/{inp}".encode()) % 1000
    case = W.make_case(f"nf_{io}_{variant}_dv{dv}", B=2, T=150, H=2, dk=64, dv=dv, io_dtype=io,
                       variant=variant, decay_scale=1.0 if variant == "decay_only" else 0.1, seed=7)
    _run(case, inp, seed)


@pytest.mark.parametrize("inp", list(POISON))
@pytest.mark.parametrize("io", ["bf16", "f32"])
def test_poisoned_input_d128(io, inp):
    # d_k = d_v = 128: the exact backward's widest per-column state gradient
    case = W.make_case(f"nf_{io}_d128", B=2, T=140, H=2, dk=128, dv=128, io_dtype=io, seed=8)
    _run(case, inp, 11 + len(inp))


@pytest.mark.parametrize("inp", ["v", "g"])
def test_poisoned_packed_dv256(inp):
    """Inside a packed batch at d_k = 128, d_v = 256 (the varlen workload's widths):
    only the poisoned sequence's stream changes class, per sequence."""
    cu = np.array([0, 70, 71, 200, 330], np.int32)
    case = W.make_case("nf_packed_dv256", B=1, T=int(cu[-1]), H=2, dk=128, dv=256, cu_seqlens=cu, seed=9)
    rng = np.random.default_rng(5)
    t, h = int(rng.integers(71, 200)), int(rng.integers(2))  # inside sequence 2
    x = getattr(case, inp)
    if x.ndim == 4:
        x[0, t, h, int(rng.integers(256))] = np.float32("nan")
    else:
        x[0, t, h] = np.float32("inf")
    dev, ref = Hn.run_device(case), Hn.run_oracle(case)
    for n, (d, r) in enumerate(zip(Hn.per_sequence(case, dev), Hn.per_sequence(case, ref))):
        res = Hn.compare(d, r)
        Hn.assert_parity(res, 1e-2, f"sequence {n}")
        if n != 2:
            for nm in ("o", "dq", "dk", "dv", "dg", "dbeta", "S_T", "dS0"):
                assert np.isfinite(d[nm]).all(), (n, nm)
        else:
            assert not np.isfinite(d["o"]).all()

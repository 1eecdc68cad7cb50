"""Tolerance-free NaN/Inf semantics of the channel-wise members.

A stream whose inputs hold a NaN or an Inf is recomputed token by token in the
channel-wise oracle's operation order (per-channel decay, erase and write), so
every output element must have the oracle's class (finite, NaN, +Inf, -Inf)
exactly, finite entries must meet the rel-L2 bar, and every other stream of the
call must stay finite.  Each case poisons one input (an element of q, k, v or
dO, one gate entry of g, b or w, one element of S0 or dS_T) for the full GDN
gates and KDA, with fp32 and bf16 activations; the workload's own injection
(NaN in v, +Inf in one g channel) runs at d_k = d_v = 128 and inside a packed
batch at d_v = 256.
"""
import zlib

import numpy as np
import pytest

import workloads as W
from tests import harness as Hn
from tests import test_gpu_cw as TC

pytestmark = pytest.mark.gpu

POISON = {"q": np.inf, "k": np.nan, "v": np.nan, "dO": -np.inf, "g": np.inf, "g_neg": -np.inf,
          "b": np.nan, "w": np.inf, "S0": np.nan, "dS_T": np.inf}


def _poison(c, inp, seed):
    rng = np.random.default_rng(seed)
    val = np.float32(POISON[inp])
    if inp in ("S0", "dS_T"):
        x = getattr(c, inp)
        n, h = int(rng.integers(x.shape[0])), int(rng.integers(c.H))
        x[n, h, int(rng.integers(c.dk)), int(rng.integers(c.dv))] = val
        return n, h
    x = getattr(c, "g" if inp == "g_neg" else inp)
    b, h = int(rng.integers(c.B)), int(rng.integers(c.H))
    t = int(rng.integers(c.T // 4, c.T))
    x[b, t, h, int(rng.integers(x.shape[-1]))] = val
    return b, h


def _run(c, stream):
    dev, ref = TC.run_device(c), TC.run_oracle(c)
    names = tuple(n for n in TC.NAMES if ref.get(n) is not None)
    res = Hn.compare(dev, ref, names=names)
    print({k: (f"{v[0]:.2e}", v[1]) for k, v in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL[c.io_dtype], c.name)
    for nm in ("o", "dq", "dk", "dv"):
        for bb in range(c.B):
            for hh in range(c.H):
                if (bb, hh) != stream:
                    assert np.isfinite(dev[nm][bb, :, hh]).all(), (nm, bb, hh)
    return dev, ref


@pytest.mark.parametrize("inp", list(POISON))
@pytest.mark.parametrize("gates", ["gbw", "kda"])
@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_poisoned_input(io, gates, inp):
    if gates == "kda" and inp in ("b", "w"):
        pytest.skip("KDA's b and w are one beta broadcast: poisoned through b/w of the full member")
    c = W.make_cw_case(f"cwnf_{io}_{gates}", 2, 150, 2, 64, 64, gates=gates, seed=13, io_dtype=io)
    stream = _poison(c, inp, zlib.crc32(f"{io}/{gates}/{inp}".encode()) % 1000)
    print("case", c.name, "poison", inp, "stream", stream, flush=True)
    dev, ref = _run(c, stream)
    poisoned = any(not np.isfinite(x).all() for x in ref.values() if x is not None)
    assert poisoned == (inp != "g_neg"), (inp, poisoned)


@pytest.mark.parametrize("gates", ["gbw", "kda"])
def test_workload_injection_d128(gates):
    """NaN in one v row and +Inf in one g channel, at d_k = d_v = 128, bf16."""
    c = W.make_cw_case(f"cwnf_inj_{gates}", 2, 200, 3, 128, 128, gates=gates, seed=17, io_dtype="bf16")
    rng = np.random.default_rng(3)
    b1, t1, h1 = 0, int(rng.integers(200)), 1
    b2, t2, h2 = 1, int(rng.integers(200)), 2
    c.v[b1, t1, h1, :] = np.float32("nan")
    c.g[b2, t2, h2, int(rng.integers(128))] = np.float32("inf")
    dev, ref = TC.run_device(c), TC.run_oracle(c)
    names = tuple(n for n in TC.NAMES if ref.get(n) is not None)
    res = Hn.compare(dev, ref, names=names)
    print({k: (f"{v[0]:.2e}", v[1]) for k, v in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL["bf16"], c.name)
    assert np.isnan(dev["o"][b1, t1:, h1]).any()
    assert np.isfinite(dev["o"][0, :, 0]).all() and np.isfinite(dev["dk"][1, :, 0]).all()


def test_packed_dv256_injection():
    cu = np.array([0, 70, 71, 200, 330], np.int32)
    c = W.make_cw_case("cwnf_packed", 1, 330, 2, 128, 256, gates="gbw", seed=19, cu_seqlens=cu, io_dtype="bf16")
    c.v[0, 150, 1, 7] = np.float32("nan")  # sequence 2, head 1
    dev, ref = TC.run_device(c), TC.run_oracle(c)
    case = W.Case("p", "gated_delta", "bf16", 1, 330, 2, 128, 256, c.q, c.k, c.v, None, None, c.S0, c.dO,
                  c.dS_T, cu_seqlens=cu)
    for n, (d, r) in enumerate(zip(Hn.per_sequence(case, dev), Hn.per_sequence(case, ref))):
        names = tuple(x for x in TC.NAMES if r.get(x) is not None)
        Hn.assert_parity(Hn.compare(d, r, names=names), 1e-2, f"sequence {n}")
        if n != 2:
            assert all(np.isfinite(d[x]).all() for x in ("o", "dq", "dk", "dv", "dS0"))

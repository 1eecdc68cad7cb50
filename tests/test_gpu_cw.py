"""Channel-wise members on the GPU against the float64 channel-wise oracle.

Every case calls the C ABI (gdn_cw_fwd / gdn_cw_bwd through the binding) on
seeded fp32 inputs and compares every output with the oracle at the fp32
bar (rel-L2 <= 1e-4 per tensor):

* full GDN gates (per-channel g, b, w), KDA (b = w = beta broadcast), GLA
  (g only), LA (no gates), each over several chunks and a ragged tail;
* d_k / d_v in {64, 128, 256} combinations, packed variable-length
  sequences (including a one-token sequence), a T shorter than one chunk;
* a strong decay (mean log-decay -4 per token and channel, within the
  documented range of the chunked kernels);
* the throughput shape (B4 T4096 H16 d128) in the launch configuration the
  bench times, checked on sampled heads;
* run-to-run bitwise determinism.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import cw_oracle as CW
from tests import harness as Hn

pytestmark = pytest.mark.gpu
TOL = Hn.TOL["f32"]
NAMES = ("o", "S_T", "states", "dq", "dk", "dv", "dg", "db", "dw", "dS0")


def _dev(x):
    return None if x is None else torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _np(x):
    return None if x is None else x.detach().cpu().numpy().astype(np.float64)


def run_device(c: W.CwCase):
    from paper_2608_12700_amd import gdn
    t = {n: _dev(getattr(c, n)) for n in ("q", "k", "v", "g", "b", "w", "S0", "dO", "dS_T")}
    cu = None if c.cu_seqlens is None else c.cu_seqlens
    o, S_T, st = gdn.cw_fwd(t["q"], t["k"], t["v"], t["g"], t["b"], t["w"], t["S0"], cu_seqlens=cu)
    r = gdn.cw_bwd(t["q"], t["k"], t["v"], t["g"], t["b"], t["w"], st, t["dO"], t["dS_T"], cu_seqlens=cu)
    torch.cuda.synchronize()
    return dict(o=_np(o), S_T=_np(S_T), states=_np(st), dq=_np(r[0]), dk=_np(r[1]), dv=_np(r[2]),
                dg=_np(r[3]), db=_np(r[4]), dw=_np(r[5]), dS0=_np(r[6]))


def run_oracle(c: W.CwCase, heads=None):
    f64 = lambda x: None if x is None else x.astype(np.float64)
    a = [f64(getattr(c, n)) for n in ("q", "k", "v", "g", "b", "w", "S0")]
    o, S_T, st = CW.cw_oracle_fwd(*a, cu_seqlens=c.cu_seqlens, heads=heads)
    r = CW.cw_oracle_bwd(*a, f64(c.dO), f64(c.dS_T), cu_seqlens=c.cu_seqlens, heads=heads)
    return dict(o=o, S_T=S_T, states=st, dq=r[0], dk=r[1], dv=r[2], dg=r[3], db=r[4], dw=r[5], dS0=r[6])


def check(c: W.CwCase, heads=None):
    print("case", c.name, c.gates, c.B, c.T, c.H, c.dk, c.dv, flush=True)
    dev = run_device(c)
    ref = run_oracle(c, heads)
    names = tuple(n for n in NAMES if ref.get(n) is not None or dev.get(n) is not None)
    res = Hn.compare(dev, ref, heads=heads, names=names)
    print(res, flush=True)
    Hn.assert_parity(res, TOL, c.name)
    return dev


@pytest.mark.parametrize("gates", ["gbw", "kda", "g", ""])
def test_members_small(gates):
    check(W.make_cw_case(f"cw_{gates or 'la'}", 2, 200, 2, 64, 64, gates=gates, seed=1))


@pytest.mark.parametrize("dk,dv", [(128, 128), (128, 64), (64, 256), (128, 256)])
def test_dims_full_gates(dk, dv):
    check(W.make_cw_case(f"cw_d{dk}_{dv}", 1, 131, 2, dk, dv, gates="gbw", seed=2))


def test_packed_sequences():
    cu = np.array([0, 70, 71, 200, 333], dtype=np.int32)
    check(W.make_cw_case("cw_packed", 1, 333, 2, 128, 128, gates="gbw", seed=3, cu_seqlens=cu))


def test_shorter_than_one_chunk():
    check(W.make_cw_case("cw_short", 3, 17, 1, 64, 128, gates="kda", seed=4))


def test_strong_decay():
    # mean log-decay about -4 per token: within 16 tokens the decay stays far
    # below the ~80 a factor of the chunked kernels can carry
    check(W.make_cw_case("cw_strong", 1, 192, 2, 128, 128, gates="gbw", seed=5, decay=5.0))


def test_throughput_shape_sampled_heads():
    c = W.make_cw_case("cw_B4_T4096_H16_d128", 4, 4096, 16, 128, 128, gates="gbw", seed=6)
    check(c, heads=[0, 11])


def test_deterministic_bitwise():
    c = W.make_cw_case("cw_det", 1, 300, 3, 128, 128, gates="gbw", seed=7)
    a, b = run_device(c), run_device(c)
    for n in NAMES:
        if a[n] is not None:
            assert np.array_equal(a[n], b[n], equal_nan=True), n

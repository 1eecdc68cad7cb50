"""HIP path vs the float64 oracle, element by element, at sizes the oracle runs
in seconds: several chunks, ragged tails, every supported (d_k, d_v), both
I/O dtypes and all three family members.  Tolerance: relative L2 <= 1e-2 per
output tensor for bf16 I/O and <= 1e-4 for fp32 I/O, plus identical
NaN/Inf class masks."""
import numpy as np
import pytest

import workloads as W
from tests import harness as Hn

pytestmark = pytest.mark.gpu


def _case(io, B, T, H, dk, dv, variant="gated_delta", **kw):
    return W.make_case(f"{io}_B{B}_T{T}_H{H}_{dk}x{dv}_{variant}", B=B, T=T, H=H, dk=dk, dv=dv,
                       io_dtype=io, variant=variant, decay_scale=1.0 if variant == "decay_only" else 0.1,
                       **kw)


CASES = [
    ("f32", 1, 256, 2, 64, 64),       # the small fp32 parity workload
    ("f32", 1, 130, 2, 128, 128),
    ("bf16", 1, 200, 2, 128, 128),
    ("bf16", 2, 130, 3, 64, 256),
    ("bf16", 1, 64, 2, 128, 64),
    ("bf16", 1, 129, 1, 64, 128),
    ("bf16", 1, 100, 2, 128, 256),
    ("f32", 2, 65, 1, 64, 128),
]


@pytest.mark.parametrize("io,B,T,H,dk,dv", CASES)
def test_parity_small(io, B, T, H, dk, dv):
    case = _case(io, B, T, H, dk, dv)
    print("case", W.describe(case), flush=True)
    res = Hn.compare(Hn.run_device(case), Hn.run_oracle(case))
    Hn.assert_parity(res, Hn.TOL[io], case.name)


@pytest.mark.parametrize("dv", [64, 128, 256])
@pytest.mark.parametrize("dk", [64, 128])
@pytest.mark.parametrize("variant", ["gated_delta", "delta", "decay_only"])
@pytest.mark.parametrize("io", ["bf16", "f32"])
def test_parity_every_instantiation(io, variant, dk, dv):
    """Every compiled (dtype, member, d_k, d_v) combination: two sequences of 130
    tokens (two whole chunks and a 2-token tail), two heads."""
    case = _case(io, 2, 130, 2, dk, dv, variant=variant, seed=dk + dv)
    print("case", W.describe(case), flush=True)
    res = Hn.compare(Hn.run_device(case), Hn.run_oracle(case))
    print({k: f"{v[0]:.2e}" for k, v in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL[io], case.name)


@pytest.mark.parametrize("variant", ["delta", "decay_only"])
@pytest.mark.parametrize("io", ["bf16", "f32"])
def test_parity_variants_small(variant, io):
    case = _case(io, 2, 150, 2, 64, 64, variant=variant)
    print("case", W.describe(case), flush=True)
    res = Hn.compare(Hn.run_device(case), Hn.run_oracle(case))
    Hn.assert_parity(res, Hn.TOL[io], case.name)


def test_parity_packed_small():
    cu = np.array([0, 5, 70, 71, 135, 135, 300], np.int32)
    case = W.make_case("bf16_packed_small", B=1, T=int(cu[-1]), H=2, dk=128, dv=64, cu_seqlens=cu)
    print("case", W.describe(case), flush=True)
    dev, ref = Hn.run_device(case), Hn.run_oracle(case)
    for n, (d, r) in enumerate(zip(Hn.per_sequence(case, dev), Hn.per_sequence(case, ref))):
        Hn.assert_parity(Hn.compare(d, r), 1e-2, f"seq {n}")

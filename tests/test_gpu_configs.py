"""HIP path vs the float64 oracle on the five specified workloads.

At full size the oracle runs on sampled (batch, head) streams: every output of
those streams is compared element by element (sequences are independent, so
a sampled stream is checked completely).  Tolerance: relative L2 <= 1e-2 per
output tensor for bf16 I/O, 1e-4 for fp32 I/O; NaN/+Inf/-Inf/finite classes
must be identical everywhere that is compared.
"""
import numpy as np
import pytest

import workloads as W
from tests import harness as Hn

pytestmark = pytest.mark.gpu


def _check(case, heads, label=None):
    print("case", W.describe(case), "heads", heads, flush=True)
    dev = Hn.run_device(case)
    ref = Hn.run_oracle(case, heads=heads)
    res = Hn.compare(dev, ref, heads=heads)
    print({k: (f"{v[0]:.2e}", v[1]) for k, v in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL[case.io_dtype], label or case.name)
    return dev, ref


def test_fp32_small_workload_full():
    _check(W.config0(), None)


def test_throughput_workload_sampled():
    _check(W.config1(), heads=[0, 9, 15])


@pytest.mark.parametrize("T", [65536, 65535, 65473])
def test_long_sequence_sampled(T):
    _check(W.config2(T), heads=[5])


@pytest.mark.parametrize("kind", ["delta", "decay_only"])
def test_family_variants_sampled(kind):
    _check(W.config3(kind), heads=[0, 17, 31])


@pytest.mark.parametrize("kind", ["nan_row", "nan_elem"])
def test_nonfinite_masks(kind):
    case = W.config3(kind)
    (b1, t1, h1, _), (b2, t2, h2) = case.injected["v_nan"], case.injected["g_inf"]
    heads = sorted({h1, h2, (h1 + 1) % case.H})
    dev, ref = _check(case, heads)
    # the poisoned streams really are poisoned, and the classes matched above
    assert np.isnan(ref["o"][b1, t1:, h1]).any()
    assert np.isnan(dev["dk"][b2, :t2, h2]).all()
    assert np.isfinite(dev["dq"][b2, :t2, h2]).all()
    # clean streams of the same batch row stay finite
    other = [h for h in heads if h not in (h1, h2)]
    for h in other:
        for nm in ("o", "dq", "dk", "dv"):
            assert np.isfinite(dev[nm][:, :, h]).all(), nm


def test_packed_varlen_per_sequence():
    case = W.config4()
    heads = [3, 12]
    print("case", W.describe(case), flush=True)
    dev = Hn.run_device(case)
    ref = Hn.run_oracle(case, heads=heads)
    for n, (d, r) in enumerate(zip(Hn.per_sequence(case, dev), Hn.per_sequence(case, ref))):
        res = Hn.compare(d, r, heads=heads)
        Hn.assert_parity(res, 1e-2, f"sequence {n}")


@pytest.mark.parametrize("io", ["bf16", "f32"])
@pytest.mark.parametrize("T", [1, 17, 63, 64, 65, 127, 129, 1000, 4095, 4097])
def test_ragged_lengths(io, T):
    case = W.make_case(f"ragged_{io}_T{T}", B=2, T=T, H=4, dk=128, dv=128, io_dtype=io)
    _check(case, heads=None if T < 1000 else [1, 2])

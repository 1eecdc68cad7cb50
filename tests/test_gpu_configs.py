"""HIP path vs the float64 oracle on the five specified workloads, in full.

Every (sequence, head) stream of every workload is compared element by
element with the token-serial oracle, which runs one stream per worker process
(``tests/oracle_pool.py``).  Tolerance: relative L2 <= 1e-2 per output tensor
for bf16 I/O, 1e-4 for fp32 I/O (per sequence for the packed workload);
NaN/+Inf/-Inf/finite classes must be identical everywhere.  The worst single
chunk of every output is reported as a diagnostic (written to
$GDN_PARITY_REPORT when set); the pass criterion is the whole-tensor figure.
"""
import numpy as np
import pytest

import workloads as W
from tests import harness as Hn
from tests import oracle_pool as OP

pytestmark = pytest.mark.gpu


def _full(case, group=None):
    print("case", W.describe(case), flush=True)
    dev = Hn.run_device(case, dtype=np.float32)
    res = OP.compare_full(case, dev)
    agg = OP.aggregate(res, group)
    worst = OP.worst_chunks(res)
    tol = Hn.TOL[case.io_dtype]
    for key, per in sorted(agg.items(), key=lambda kv: str(kv[0])):
        print(key, {k: (f"{v[0]:.2e}", v[1]) for k, v in per.items()}, flush=True)
    print("worst chunk:", {k: f"{v['rel']:.2e}@(seq {v['sequence']}, head {v['head']}, chunk {v['chunk']})"
                           for k, v in worst.items()}, flush=True)
    OP.write_report(case.name, dict(case=W.describe(case), tolerance=tol,
                                    rel_l2={str(k): {n: v[0] for n, v in per.items()} for k, per in agg.items()},
                                    classes_equal=all(v[1] for per in agg.values() for v in per.values()),
                                    worst_chunk=worst))
    for key, per in agg.items():
        Hn.assert_parity(per, tol, f"{case.name} {key}")
    return dev, agg


def test_fp32_small_workload_full():
    _full(W.config0())


@pytest.mark.timeout(600)
def test_throughput_workload_full():
    _full(W.config1())


@pytest.mark.timeout(900)
@pytest.mark.parametrize("T", [65536, 65535, 65473])
def test_long_sequence_full(T):
    _full(W.config2(T))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("kind", ["delta", "decay_only"])
def test_family_variants_full(kind):
    _full(W.config3(kind))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("kind", ["nan_row", "nan_elem"])
def test_nonfinite_masks_full(kind):
    case = W.config3(kind)
    (b1, t1, h1, _), (b2, t2, h2) = case.injected["v_nan"], case.injected["g_inf"]
    dev, _ = _full(case)
    # the poisoned streams really are poisoned (the classes matched the oracle above)
    assert np.isnan(dev["o"][b1, t1:, h1]).any()
    assert np.isnan(dev["dk"][b2, :t2, h2]).all()
    assert np.isfinite(dev["dq"][b2, :t2, h2]).all()
    # every other stream stays finite
    mask = np.ones((case.B, case.H), bool)
    mask[b1, h1] = mask[b2, h2] = False
    for nm in ("o", "dq", "dk", "dv"):
        x = np.moveaxis(dev[nm], 2, 1)[mask]
        assert np.isfinite(x).all(), nm


@pytest.mark.timeout(900)
def test_packed_varlen_per_sequence_full():
    _full(W.config4(), group=lambda r: r["n"])


@pytest.mark.parametrize("io", ["bf16", "f32"])
@pytest.mark.parametrize("T", [1, 17, 63, 64, 65, 127, 129, 1000, 4095, 4097])
def test_ragged_lengths(io, T):
    case = W.make_case(f"ragged_{io}_T{T}", B=2, T=T, H=4, dk=128, dv=128, io_dtype=io)
    print("case", W.describe(case), flush=True)
    if T < 1000:
        res = Hn.compare(Hn.run_device(case), Hn.run_oracle(case))
        Hn.assert_parity(res, Hn.TOL[io], case.name)
    else:
        _full(case)

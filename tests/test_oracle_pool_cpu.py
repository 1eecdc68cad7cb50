"""The whole-workload comparison machinery (tests/oracle_pool.py) on the CPU.

Stand-in "device" outputs are the oracle's own results rounded to float32,
then perturbed: the per-stream sums aggregated by the pool must give the same
relative L2 and class verdicts as a direct comparison of the full tensors
(harness.compare), per sequence for packed batches, and the worst-chunk report
must point at a chunk that was perturbed on purpose.
"""
import numpy as np
import pytest

import workloads as W
from tests import harness as Hn
from tests import oracle_pool as OP


def _fake_device(case, seed=1, scale=1e-3):
    ref = Hn.run_oracle(case)
    rng = np.random.default_rng(seed)
    dev = {}
    for nm, y in ref.items():
        if y is None:
            continue
        x = y * (1 + scale * rng.standard_normal(y.shape))
        dev[nm] = x.astype(np.float32)
    return ref, dev


@pytest.mark.parametrize("packed", [False, True])
def test_pool_matches_direct_comparison(packed):
    if packed:
        cu = np.array([0, 70, 70, 200], np.int32)
        case = W.make_case("pool_packed", B=1, T=200, H=3, dk=16, dv=8, io_dtype="f32", cu_seqlens=cu)
    else:
        case = W.make_case("pool", B=2, T=150, H=3, dk=16, dv=8, io_dtype="f32")
    ref, dev = _fake_device(case)
    res = OP.compare_full(case, dev)
    assert len(res) == case.N * case.H
    agg = OP.aggregate(res)["all"]
    direct = Hn.compare({k: v.astype(np.float64) for k, v in dev.items()}, ref)
    for nm, (rel, ok, cnt) in direct.items():
        assert agg[nm][1] == ok and agg[nm][0] == pytest.approx(rel, rel=1e-9), nm
    if packed:
        per = OP.aggregate(res, group=lambda r: r["n"])
        assert set(per) == {0, 1, 2}
        d1 = Hn.per_sequence(case, {k: v.astype(np.float64) for k, v in dev.items()})[2]
        r1 = Hn.per_sequence(case, ref)[2]
        direct = Hn.compare(d1, r1)
        for nm, (rel, ok, cnt) in direct.items():
            assert per[2][nm][0] == pytest.approx(rel, rel=1e-9), nm


def test_pool_sees_a_bad_chunk_and_a_class_change():
    case = W.make_case("pool_bad", B=2, T=200, H=3, dk=16, dv=8, io_dtype="f32")
    ref, dev = _fake_device(case, scale=1e-6)
    dev["dk"][1, 130:140, 2] *= 1.5          # chunk 2 of stream (b=1, h=2)
    dev["dq"][0, 5, 1, 3] = np.float32("inf")  # one class change
    res = OP.compare_full(case, dev)
    agg = OP.aggregate(res)["all"]
    w = OP.worst_chunks(res)
    assert w["dk"]["sequence"] == 1 and w["dk"]["head"] == 2 and w["dk"]["chunk"] == 2
    assert w["dk"]["rel"] > 0.1
    assert not agg["dq"][1] and agg["dk"][1]
    assert agg["o"][0] < 1e-5


def test_zero_reference_needs_zero_device():
    # head 1 has v = 0 and S0 = 0: its o, S_T and chunk states are exactly zero
    case = W.make_case("pool_zero", B=1, T=70, H=2, dk=16, dv=8, io_dtype="f32", S0_std=0.0)
    case.v[:, :, 1] = 0
    ref, dev = _fake_device(case, scale=0.0)
    by_head = lambda r: r["h"]
    agg = OP.aggregate(OP.compare_full(case, dev), group=by_head)
    assert agg[1]["o"][0] == 0.0 and agg[1]["states"][0] == 0.0
    dev["o"][0, 33, 1, 2] = 1e-30
    agg = OP.aggregate(OP.compare_full(case, dev), group=by_head)
    assert agg[1]["o"][0] == float("inf") and agg[0]["o"][0] < 1e-6

"""Shared helpers for the GPU parity tests: run a seeded case on the HIP path
and on the float64 oracle, and compare them (rel-L2 over entries finite in
both, plus exact equality of the NaN/+Inf/-Inf/finite class of every entry).
"""
from __future__ import annotations

import numpy as np

import workloads as W
from oracle import gdn_oracle as O

OUT_NAMES = ("o", "S_T", "states", "dq", "dk", "dv", "dg", "dbeta", "dS0")
TOL = {"bf16": 1e-2, "f32": 1e-4}


def device_inputs(case: W.Case, device="cuda"):
    import torch
    dt = torch.bfloat16 if case.io_dtype == "bf16" else torch.float32

    def act(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(device=device, dtype=dt)

    def f32(x):
        return None if x is None else torch.from_numpy(np.ascontiguousarray(x)).to(device)

    return dict(q=act(case.q), k=act(case.k), v=act(case.v), g=f32(case.g), beta=f32(case.beta),
                S0=f32(case.S0), dO=act(case.dO), dS_T=f32(case.dS_T))


def run_device(case: W.Case, device="cuda", keep_torch=False, dtype=np.float64):
    """Forward then backward on the HIP path; returns numpy outputs (float64 by
    default; float32 holds every device value exactly too)."""
    import torch
    from paper_2608_12700_amd import gdn
    t = device_inputs(case, device)
    cu = None if case.cu_seqlens is None else gdn.Packed(case.cu_seqlens, device)
    o, S_T, st = gdn.fwd(t["q"], t["k"], t["v"], t["g"], t["beta"], t["S0"], variant=case.variant,
                         cu_seqlens=cu)
    dq, dk, dv, dg, db, dS0 = gdn.bwd(t["q"], t["k"], t["v"], t["g"], t["beta"], st, t["dO"],
                                      t["dS_T"], variant=case.variant, cu_seqlens=cu)
    torch.cuda.synchronize()
    outs = dict(o=o, S_T=S_T, states=st, dq=dq, dk=dk, dv=dv, dg=dg, dbeta=db, dS0=dS0)
    if keep_torch:
        return outs
    return {k: (None if x is None else x.float().cpu().numpy().astype(dtype, copy=False)) for k, x in outs.items()}


def run_oracle(case: W.Case, heads=None):
    f = lambda x: None if x is None else x.astype(np.float64)
    q, k, v, g, b = f(case.q), f(case.k), f(case.v), f(case.g), f(case.beta)
    S0, dO, dST = f(case.S0), f(case.dO), f(case.dS_T)
    o, S_T, st = O.oracle_fwd(q, k, v, g, b, S0, variant=case.variant, cu_seqlens=case.cu_seqlens,
                              heads=heads)
    dq, dk, dv, dg, db, dS0 = O.oracle_bwd(q, k, v, g, b, S0, dO, dST, variant=case.variant,
                                           cu_seqlens=case.cu_seqlens, heads=heads)
    return dict(o=o, S_T=S_T, states=st, dq=dq, dk=dk, dv=dv, dg=dg, dbeta=db, dS0=dS0)


def _head_axis(name):
    # q/k/v/o/dq/dk/dv: [B,T,H,d] -> 2 ; g/beta: [B,T,H] -> 2 ; states/S: [*,H,dk,dv] -> 1
    return 1 if name in ("S_T", "states", "dS0") else 2


def select(name, x, heads):
    if heads is None or x is None:
        return x
    return np.take(x, heads, axis=_head_axis(name))


def classes(x):
    c = np.zeros(x.shape, np.int8)
    c[np.isnan(x)] = 1
    c[np.isposinf(x)] = 2
    c[np.isneginf(x)] = 3
    return c


def compare(dev: dict, ref: dict, heads=None, names=OUT_NAMES):
    """Per output: (rel_l2 over jointly finite entries, classes equal, count)."""
    res = {}
    for nm in names:
        x, y = dev.get(nm), ref.get(nm)
        if x is None and y is None:
            continue
        assert x is not None and y is not None, nm
        x, y = select(nm, x, heads), select(nm, y, heads)
        assert x.shape == y.shape, (nm, x.shape, y.shape)
        cls_ok = bool(np.array_equal(classes(x), classes(y)))
        m = np.isfinite(x) & np.isfinite(y)
        ny = np.linalg.norm(y[m])
        err = np.linalg.norm(x[m] - y[m])
        if ny > 0:
            rel = float(err / ny)
        else:
            # an all-zero reference must be met exactly: any nonzero entry fails
            rel = 0.0 if not np.any(x[m]) else float("inf")
        res[nm] = (rel, cls_ok, int(m.sum()))
    return res


def assert_parity(res: dict, tol: float, label=""):
    bad = {k: v for k, v in res.items() if not (v[0] <= tol and v[1])}
    assert not bad, f"{label}: parity failed {bad} (all: {res})"


def per_sequence(case: W.Case, arrs: dict):
    """Split packed outputs per sequence: list of dicts."""
    out = []
    off = 0
    for n, (_, s, L) in enumerate(case.seq_bounds()):
        nt = -(-L // case.chunk)
        d = {}
        for nm, x in arrs.items():
            if x is None:
                continue
            if nm in ("S_T", "dS0"):
                d[nm] = x[n:n + 1]
            elif nm == "states":
                d[nm] = x[off:off + nt]
            else:
                d[nm] = x[:, s:s + L]
        out.append(d)
        off += nt
    return out

"""Whole-workload comparisons of the HIP path with the float64 oracle.

The oracle is token-serial and runs one (sequence, head) stream per worker
process; a full workload (up to 16 heads x 65536 tokens) then takes seconds to
tens of seconds on the host's cores.  The worker pool is forked once, from
``tests/conftest.py`` before anything touches the GPU, so no worker is a copy
of a process that holds a GPU context.  Inputs and device outputs go to the
workers through ``.npy`` files in a temporary directory (``/dev/shm`` when
present) that they map read-only; each worker returns per-output sums for its
stream only, so nothing large travels back:

  err2, ref2    squared L2 norms of (device - oracle) and of the oracle over the
                entries finite in both;
  dev2          squared norm of the device entries there (for all-zero references);
  mismatch      entries whose class (finite, NaN, +Inf, -Inf) differs;
  worst         the worst relative L2 of one 64-token chunk (one chunk state,
                or the whole stream for S_T and dS0), with its chunk index.

Whole-tensor relative L2 is sqrt(sum err2 / sum ref2): the same number as a
comparison of the full tensors.
"""
from __future__ import annotations

import json
import multiprocessing as mp
import os
import shutil
import tempfile

import numpy as np

_POOL = None
NAMES = ("o", "S_T", "states", "dq", "dk", "dv", "dg", "dbeta", "dS0")
PER_TOKEN = ("o", "dq", "dk", "dv", "dg", "dbeta")


def workers() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(n, 16))


def start():
    """Fork the pool (call before any GPU use in this process)."""
    global _POOL
    if _POOL is None:
        _POOL = mp.get_context("fork").Pool(workers(), initializer=_init_worker)
    return _POOL


def pool():
    return _POOL if _POOL is not None else start()


def close():
    global _POOL
    if _POOL is not None:
        _POOL.terminate()
        _POOL = None


def _init_worker():
    os.environ["OMP_NUM_THREADS"] = os.environ["OPENBLAS_NUM_THREADS"] = "1"
    os.environ["MKL_NUM_THREADS"] = "1"


def _classes(x):
    c = np.zeros(x.shape, np.int8)
    c[np.isnan(x)] = 1
    c[np.isposinf(x)] = 2
    c[np.isneginf(x)] = 3
    return c


def _rel(x, y):
    m = np.isfinite(x) & np.isfinite(y)
    ny = float(np.sum(y[m] ** 2))
    ne = float(np.sum((x[m] - y[m]) ** 2))
    if ny > 0:
        return (ne / ny) ** 0.5
    return 0.0 if not np.any(x[m]) else float("inf")


def _stats(x, y, chunk_axis_len):
    """Sums for one output of one stream; chunks of chunk_axis_len rows along axis 0."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    m = np.isfinite(x) & np.isfinite(y)
    out = dict(err2=float(np.sum((x[m] - y[m]) ** 2)), ref2=float(np.sum(y[m] ** 2)),
               dev2=float(np.sum(x[m] ** 2)), mismatch=int(np.sum(_classes(x) != _classes(y))),
               count=int(x.size), worst=0.0, worst_chunk=0)
    n = x.shape[0] if x.ndim else 1
    step = chunk_axis_len or max(n, 1)
    for c, i in enumerate(range(0, max(n, 1), step)):
        r = _rel(x[i:i + step], y[i:i + step])
        if r > out["worst"]:
            out["worst"], out["worst_chunk"] = r, c
    return out


def _stream_job(job):
    from oracle import gdn_oracle as O
    d = job["dir"]
    b, s, L, h, n, off = job["b"], job["s"], job["L"], job["h"], job["n"], job["off"]
    chunk, variant = job["chunk"], job["variant"]

    def arr(name):
        p = os.path.join(d, name + ".npy")
        return np.load(p, mmap_mode="r") if os.path.exists(p) else None

    def tok(name):
        a = arr(name)
        return None if a is None else np.asarray(a[b, s:s + L, h], dtype=np.float64)[None]

    q, k, v, g, beta, dO = (tok(x) for x in ("q", "k", "v", "g", "beta", "dO"))
    S0 = np.asarray(arr("S0")[n, h], dtype=np.float64)[None]
    dST = np.asarray(arr("dS_T")[n, h], dtype=np.float64)[None]
    o, S_T, st = O.fwd_streams(q, k, v, g, beta, S0, variant, chunk)
    dq, dk, dv, dg, db, dS0 = O.bwd_streams(q, k, v, g, beta, S0, dO, dST, variant, chunk)
    ref = dict(o=o[0], S_T=S_T[0], states=st[0], dq=dq[0], dk=dk[0], dv=dv[0],
               dg=None if dg is None else dg[0], dbeta=None if db is None else db[0], dS0=dS0[0])
    nt = st.shape[1]
    res = {}
    for nm in NAMES:
        y = ref[nm]
        a = arr("dev_" + nm)
        if y is None or a is None:
            continue
        if nm in PER_TOKEN:
            x, cl = a[b, s:s + L, h], chunk
        elif nm == "states":
            x, cl = a[off:off + nt, h], 1
        else:
            x, cl = a[n, h], 0
        res[nm] = _stats(x, y, cl)
    return dict(n=n, b=b, h=h, stats=res)


def stream_specs(case):
    """(n, batch row, first token, length, first chunk-state entry) per sequence."""
    specs, off = [], 0
    for n, (b, s, L) in enumerate(case.seq_bounds()):
        specs.append((n, b, s, L, off))
        off += -(-L // case.chunk)
    return specs


def compare_full(case, dev: dict, heads=None, log=print):
    """Every (sequence, head) stream of ``case`` against the oracle.  ``dev`` maps
    output names to numpy arrays in the API layout.  Returns the per-stream
    results (see the module doc)."""
    root = "/dev/shm" if os.path.isdir("/dev/shm") else None
    d = tempfile.mkdtemp(prefix="gdn_parity_", dir=root)
    try:
        for nm in ("q", "k", "v", "g", "beta", "S0", "dO", "dS_T"):
            x = getattr(case, nm)
            if x is not None:
                np.save(os.path.join(d, nm + ".npy"), np.ascontiguousarray(x, dtype=np.float32))
        for nm in NAMES:
            x = dev.get(nm)
            if x is not None:
                np.save(os.path.join(d, "dev_" + nm + ".npy"), np.ascontiguousarray(x, dtype=np.float32))
        hs = range(case.H) if heads is None else heads
        jobs = [dict(dir=d, b=b, s=s, L=L, h=h, n=n, off=off, chunk=case.chunk, variant=case.variant)
                for (n, b, s, L, off) in stream_specs(case) for h in hs]
        # longest streams first, so the pool's tail is short
        jobs.sort(key=lambda j: -j["L"])
        out = []
        for i, r in enumerate(pool().imap_unordered(_stream_job, jobs, chunksize=1)):
            out.append(r)
            if (i + 1) % max(1, len(jobs) // 4) == 0:
                log(f"  oracle: {i + 1}/{len(jobs)} streams", flush=True)
        return out
    finally:
        shutil.rmtree(d, ignore_errors=True)


def aggregate(results, group=None):
    """Whole-tensor figures per output (per group key if ``group`` maps a result
    to one, e.g. the sequence index): {key: {name: (rel, classes_equal, count)}}."""
    acc = {}
    for r in results:
        key = group(r) if group else "all"
        for nm, st in r["stats"].items():
            a = acc.setdefault(key, {}).setdefault(nm, dict(err2=0.0, ref2=0.0, dev2=0.0, mismatch=0, count=0))
            for f in ("err2", "ref2", "dev2", "mismatch", "count"):
                a[f] += st[f]
    out = {}
    for key, per in acc.items():
        out[key] = {}
        for nm, a in per.items():
            if a["ref2"] > 0:
                rel = (a["err2"] / a["ref2"]) ** 0.5
            else:
                rel = 0.0 if a["dev2"] == 0 else float("inf")
            out[key][nm] = (rel, a["mismatch"] == 0, a["count"])
    return out


def worst_chunks(results):
    """Per output: the worst single-chunk relative L2 over every stream, and where."""
    w = {}
    for r in results:
        for nm, st in r["stats"].items():
            if nm not in w or st["worst"] > w[nm]["rel"]:
                w[nm] = dict(rel=st["worst"], sequence=r["n"], head=r["h"], chunk=st["worst_chunk"])
    return w


def write_report(name, summary: dict):
    """Adds one case's figures to $GDN_PARITY_REPORT/<name>.json when set."""
    d = os.environ.get("GDN_PARITY_REPORT")
    if not d:
        return
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, name + ".json"), "w") as fh:
        json.dump(summary, fh, indent=1, default=float)

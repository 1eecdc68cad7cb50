#!/usr/bin/env python3
"""Throughput of the gated-delta-rule forward + training backward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

One step = gdn_fwd then gdn_bwd (the whole hot path) over one batch of the
throughput workload: bf16 I/O with fp32 gates and states, B=4, T=4096, H=16,
d_k=d_v=128, chunk 64, seeded synthetic inputs already resident in HBM.
Outputs and workspaces are allocated once, outside the timed region.  The
reported step time is the mean over K steps that each start with cold caches
(a 512 MiB scratch write before every step, outside its event interval); the
same K steps run back to back are reported beside it.

The JSON line carries, besides tokens/s:
  roofline      the training backward (gdn_bwd), whose binding roofline is
                HBM: its compulsory bytes (every tensor of the call read or
                written once at its dtype, 2,832 B per token-head here; workspace
                traffic is not counted) divided by its duration, measured live
                with HIP events recorded on the launch stream around each stage
                of the timed steps, against MI355X's 8 TB/s HBM peak.  The
                dominant kernel (the chunk-gradient kernel) is reported inside
                it on the same basis, and as kernel_io_frac on its own inputs
                and outputs including workspace operands;
  cpu_baseline  the float64 oracle (fwd + bwd) on the host cores, on a bounded
                sample of the same workload's (b, h) streams.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
CH = 64
ROOT = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_bf16_B4_T4096_H16_d128.json")
CW_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_cw_bf16_B4_T4096_H16_d128.json")
STAGE_OF_KERNEL = {"k_prep_fwd": "fwd_prep", "k_scan_fwd": "fwd_scan", "k_prep_bwd": "bwd_prep",
                   "k_scan_bwd": "bwd_scan", "k_grad_bf": "bwd_grad"}


def cw_stage_of(name: str):
    """Stage of a channel-wise kernel name (mangled or demangled), or None."""
    if "k_cw_prep" in name:
        return "cw_bwd_prep" if ("true>" in name or "Lb1E" in name) else "cw_fwd_prep"
    for k, st in (("k_scan_fwd", "cw_fwd_scan"), ("k_scan_bwd", "cw_bwd_scan"),
                  ("k_cw_grad_v", "cw_bwd_grad_v"), ("k_cw_grad_d", "cw_bwd_grad_d")):
        if k in name:
            return st
    return None
COPY_BYTES = 256 * 1024 * 1024


def source_digest() -> str:
    """Digest of every kernel source: measured traffic is reported only while it matches."""
    import hashlib
    d = os.path.join(ROOT, "paper_2608_12700_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f.endswith((".hpp", ".hip", ".cpp", ".h")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(stage: str, path: str = TRAFFIC_FILE):
    """HBM bytes per launch of `stage` from the committed counter summary, or None
    when there is none or the kernels changed since it was taken."""
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != source_digest():
        return None
    k = t.get("kernels", {}).get(stage)
    return None if k is None else k["hbm_bytes_per_launch"]


def _counter_rows(d):
    import csv
    import glob
    out = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            out += list(csv.DictReader(fh))
    return out


def summarize_counters(fetch_dir, write_dir, calib_fetch_dir, calib_write_dir, command, cw=False, cw_es=2):
    """Turn FETCH_SIZE / WRITE_SIZE passes (KiB per dispatch) over the bench and
    over a plain copy of COPY_BYTES into HBM bytes per launch of each stage."""
    def stage_of(name):
        if cw:
            return cw_stage_of(name)
        for k, st in STAGE_OF_KERNEL.items():
            if k in name:
                return st
        return None

    def per_kernel(d, counter):
        acc = {}
        for r in _counter_rows(d):
            if r["Counter_Name"] != counter:
                continue
            st = stage_of(r["Kernel_Name"])
            if st is not None:
                acc.setdefault(st, []).append(float(r["Counter_Value"]))
        return {st: sum(v) / len(v) for st, v in acc.items()}

    def copy_kib(d, counter):
        vals = [float(r["Counter_Value"]) for r in _counter_rows(d) if r["Counter_Name"] == counter]
        return max(vals)  # the copy is the largest dispatch of the calibration run
    fscale = COPY_BYTES / 1024.0 / copy_kib(calib_fetch_dir, "FETCH_SIZE")
    wscale = COPY_BYTES / 1024.0 / copy_kib(calib_write_dir, "WRITE_SIZE")
    f, w = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    km = cw_kernel_model(4, 4096, 16, 128, 128, es=cw_es) if cw else kernel_model(4, 4096, 16, 128, 128, 2)
    kern = {}
    for st in sorted(f):
        b = (f[st] * fscale + w.get(st, 0.0) * wscale) * 1024.0
        kern[st] = {"fetch_kib": round(f[st], 1), "write_kib": round(w.get(st, 0.0), 1),
                    "hbm_bytes_per_launch": int(b), "algorithmic_bytes_per_launch": int(km[st][0]),
                    "ratio": round(b / km[st][0], 3)}
    return {"source_digest": source_digest(), "command": command,
            "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
            "calibration": f"plain device copy of {COPY_BYTES} bytes (bench.py --copy-kernel)",
            "kernels": kern}


SQ_FILE = os.path.join(ROOT, "profiles", "sq_counters_bf16_B4_T4096_H16_d128.json")


def summarize_sq(dirs, command):
    """Per stage of the metric workload: SQ instruction counters from rocprofv3
    --pmc passes (one folder per pass), averaged over dispatches, as totals per
    launch and per wave; plus the ratios the kernel designs are judged by."""
    acc = {}
    for d in dirs:
        for r in _counter_rows(d):
            st = None
            for k, stg in STAGE_OF_KERNEL.items():
                if k in r["Kernel_Name"]:
                    st = stg
            if st is None:
                continue
            acc.setdefault(st, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    km = kernel_model(4, 4096, 16, 128, 128, 2)
    out = {}
    for st, cs in sorted(acc.items()):
        avg = {c: sum(v) / len(v) for c, v in cs.items()}
        waves = avg.get("SQ_WAVES", 0.0)
        e = {"per_launch": {c: round(x) for c, x in avg.items()}}
        if waves:
            e["per_wave"] = {c: round(x / waves, 1) for c, x in avg.items()
                             if c.startswith("SQ_INSTS") or c.startswith("SQ_LDS")}
        if avg.get("SQ_INSTS_MFMA"):
            e["valu_per_mfma"] = round(avg.get("SQ_INSTS_VALU", 0.0) / avg["SQ_INSTS_MFMA"], 2)
        if avg.get("SQ_ACTIVE_INST_LDS"):
            e["lds_bank_conflict_per_lds_active_cycle"] = round(
                avg.get("SQ_LDS_BANK_CONFLICT", 0.0) / avg["SQ_ACTIVE_INST_LDS"], 3)
        if avg.get("SQ_BUSY_CYCLES"):
            e["valu_mfma_busy_per_busy_cycle"] = round(avg.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / avg["SQ_BUSY_CYCLES"], 4)
        if st in km:
            e["model_flops_per_launch"] = int(km[st][1])
        out[st] = e
    return {"source_digest": source_digest(), "command": command,
            "note": "SQ_* counters summed over the device per dispatch (rocprofv3 --pmc), averaged over the "
                    "dispatches of the run; per_wave = per launch / SQ_WAVES",
            "stages": out}


def summarize_trace(trace_dir, command, title="gated delta rule fwd+bwd, bf16 I/O, B=4 T=4096 H=16 dk=dv=128"):
    """Markdown table of a `rocprofv3 --kernel-trace --stats --output-format csv` run."""
    import csv
    import glob
    import re
    f = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)[0]
    with open(f) as fh:
        rows = list(csv.DictReader(fh))

    def short(n):
        d = re.search(r"gdn::(k_\w+)<([^>]*)>", n)  # demangled name
        if d:
            args = [x.strip() for x in d.group(2).split(",")]
            nums = [x for x in args if x.isdigit()][:2]
            mode = " (bwd)" if d.group(1) == "k_cw_prep" and args[-1] == "true" else ""
            bf = " bf16" if "bf16" in args or "__hip_bfloat16" in d.group(2) else ""
            return f"{d.group(1)}<{','.join(nums)}>" + bf + mode
        m = re.search(r"gdn\d*(k_\w+?)I(.*?)EE", n)
        if not m:
            return n[:60]
        nums = re.findall(r"Li(\d+)E", m.group(2))
        flags = re.findall(r"Lb([01])E", m.group(2))
        mode = " (bwd)" if m.group(1) == "k_cw_prep" and flags == ["1"] else ""
        return f"{m.group(1)}<{','.join(nums)}>" + (" bf16" if "DF16b" in m.group(2) else "") + mode
    out = [f"# Kernel trace: {title}", "",
           "Command (from the repository root, one MI355X):", "", "```", command, "```", "",
           "| kernel | calls | average (us) | total (us) | % |", "|---|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        if float(r["Percentage"]) < 0.2:
            continue
        out.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['TotalDurationNs']) / 1e3:.1f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out) + "\n"


def copy_kernel():
    """A plain device copy of COPY_BYTES, three times: the counter calibration run."""
    import torch
    a_ = torch.randn(COPY_BYTES // 4, device="cuda")
    b_ = torch.empty_like(a_)
    torch.cuda.synchronize()
    for _ in range(3):
        b_.copy_(a_)
    torch.cuda.synchronize()
    print(f"copied {COPY_BYTES} bytes x3", flush=True)


def kernel_model(B, T, H, dk, dv, es, N=None, nch=None):
    """Algorithmic bytes and flops per launch of every stage (compulsory traffic
    of the kernel's own inputs and outputs, each moved once at its stored dtype).
    """
    N = B if N is None else N
    nch = B * (-(-T // CH)) if nch is None else nch
    tiles = nch * H
    g4 = 4 * CH  # one fp32 per token of a chunk
    st = dk * dv * 4
    qk = CH * dk * es  # one chunk of q or k (or a 64 x dk operand) in the I/O dtype
    vv = CH * dv * es  # one chunk of v, o, dO (or a 64 x dv operand)
    pp = CH * CH * es  # one 64 x 64 operand
    per = {
        # q, k, v, g, beta -> gcum, W, U, Khat^T, P
        "fwd_prep": (2 * qk + vv + 2 * g4 + g4 + 2 * qk + vv + pp,
                     3 * 2 * CH * CH * dk + CH ** 3 / 3 + 2 * CH * CH * dk + 2 * CH * CH * dv),
        # q, W, Khat^T, P, U, gcum -> chunk states, o
        "fwd_scan": (3 * qk + pp + vv + g4 + st + vv,
                     3 * 2 * CH * dk * dv + 2 * CH * CH * dv),
        # q, k, g, beta -> gcum, W^T, (diag(e^G) Q)^T, P^T, T
        "bwd_prep": (2 * qk + 2 * g4 + g4 + 2 * qk + 2 * pp,
                     3 * 2 * CH * CH * dk + CH ** 3 / 3),
        # k, gcum, W^T, Qg^T, dO, P^T -> dh (I/O dtype), dU'^T
        "bwd_scan": (3 * qk + g4 + vv + pp + dk * dv * es + vv,
                     3 * 2 * CH * dk * dv + 2 * CH * CH * dv),
        # q, k, v, g, beta, T, states, dO, dh, dU'^T -> dq, dk, dv, dg, dbeta
        "bwd_grad": (2 * qk + vv + 2 * g4 + pp + st + vv + dk * dv * es + vv + 2 * qk + vv + 2 * g4,
                     5 * 2 * CH * CH * dk + CH ** 3 / 3 + 4 * CH ** 3 + 5 * 2 * CH * dk * dv
                     + 5 * 2 * CH * CH * dv),
    }
    out = {k: (b * tiles, f * tiles) for k, (b, f) in per.items()}
    sio = 2 * N * H * dk * dv * 4  # S0 / S_T or dS_T / dS0
    out["fwd_scan"] = (out["fwd_scan"][0] + sio, out["fwd_scan"][1])
    out["bwd_scan"] = (out["bwd_scan"][0] + sio, out["bwd_scan"][1])
    return out


def cw_kernel_model(B, T, H, dk, dv, N=None, es=4):
    """Algorithmic bytes and flops per launch of the channel-wise stages (each
    kernel's own inputs and outputs moved once; the activations q, k, v, o, dO
    and their gradients, and the operands the scans read or write (P, e^G Q,
    Khat, W, U, dO^T, dh, dU'^T), at es bytes; everything else fp32)."""
    N = B if N is None else N
    tiles = B * (-(-T // CH)) * H
    ck, cv, cc, st, vk = CH * dk * 4, CH * dv * 4, CH * CH * 4, dk * dv * 4, dk * 4
    ak, av = CH * dk * es, CH * dv * es  # activation tiles
    ok, ov, oc, ost = CH * dk * es, CH * dv * es, CH * CH * es, dk * dv * es  # scan operands
    per = {
        # q, k, g, b, v, w -> G_last, P, e^G Q, Khat^T, W, U
        "cw_fwd_prep": (2 * ak + 2 * ck + av + cv + vk + oc + 3 * ok + ov,
                        2 * 2 * CH * CH * dk + CH ** 3 / 3 + 2 * CH * CH * dk + 2 * CH * CH * dv),
        # e^G Q, W, Khat^T, P, U, G_last -> chunk states, o
        "cw_fwd_scan": (3 * ok + oc + ov + vk + st + av, 3 * 2 * CH * dk * dv + 2 * CH * CH * dv),
        # q, k, g, b, dO -> G_last, P^T, T, (e^G Q)^T, Khat, W^T, Gamma*b*k, dO^T
        "cw_bwd_prep": (2 * ak + 2 * ck + av + vk + oc + cc + 3 * ok + ck + ov,
                        2 * 2 * CH * CH * dk + CH ** 3 / 3 + 2 * CH * CH * dk),
        # Khat, W^T, (e^G Q)^T, dO^T, P^T, G_last -> dh, dU'^T
        "cw_bwd_scan": (3 * ok + ov + oc + vk + ost + ov, 3 * 2 * CH * dk * dv + 2 * CH * CH * dv),
        # v, w, dO, state, T, Gamma*b*k, dh, dU'^T -> dv, dw, dP, dA, X, dQg, dKhat, <h, dh>
        "cw_bwd_grad_v": (2 * av + cv + st + cc + ck + ost + ov + av + cv + 2 * cc + 3 * ck + vk,
                          2 * CH * dk * dv + 3 * 2 * CH * CH * dv + 3 * 2 * CH * dk * dv),
        # q, k, g, b, dP, dA, X, dQg, dKhat, <h, dh> -> dq, dk, dg, db
        "cw_bwd_grad_d": (2 * ak + 2 * ck + 2 * cc + 3 * ck + vk + 2 * ak + 2 * ck, 4 * 2 * CH * CH * dk),
    }
    out = {k: (b * tiles, f * tiles) for k, (b, f) in per.items()}
    sio = 2 * N * H * dk * dv * 4
    out["cw_fwd_scan"] = (out["cw_fwd_scan"][0] + sio, out["cw_fwd_scan"][1])
    out["cw_bwd_scan"] = (out["cw_bwd_scan"][0] + sio, out["cw_bwd_scan"][1])
    return out


def _cw_oracle_stream(args):
    """One (b, h) stream of the channel-wise oracle: backward (which runs the forward)."""
    os.environ["OMP_NUM_THREADS"] = os.environ["OPENBLAS_NUM_THREADS"] = "1"
    os.environ["MKL_NUM_THREADS"] = "1"
    import numpy as np
    from oracle import cw_oracle as CWO
    q, k, v, g, b, w, S0, dO, dST = args
    f = lambda x: None if x is None else x[None].astype(np.float64)
    CWO.cw_fwd_streams(f(q), f(k), f(v), f(g), f(b), f(w), f(S0))
    CWO.cw_bwd_streams(f(q), f(k), f(v), f(g), f(b), f(w), f(S0), f(dO), f(dST))
    return q.shape[0]


def cw_cpu_baseline(case, budget_s=15.0):
    """The channel-wise oracle on a bounded sample of the workload's streams, all host cores."""
    import multiprocessing as mp
    cores, affinity = host_workers()
    streams = [(b, h) for b in range(case.B) for h in range(case.H)]
    per_stream_s = 3.0 * (case.T / 4096) * (case.dk * case.dv / 16384)
    n = min(len(streams), int(max(cores, budget_s * cores / per_stream_s)))
    sl = lambda x, b, h: None if x is None else x[b, :, h]
    tasks = [(sl(case.q, b, h), sl(case.k, b, h), sl(case.v, b, h), sl(case.g, b, h), sl(case.b, b, h),
              sl(case.w, b, h), case.S0[b, h], sl(case.dO, b, h), case.dS_T[b, h]) for (b, h) in streams[:n]]
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        done = sum(pool.map(_cw_oracle_stream, tasks, chunksize=1))
    wall = time.perf_counter() - t0
    return {"value": round(done / case.H / wall, 1), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": (f"{n} of {len(streams)} (b,h) streams, full T={case.T} each, float64 token-serial fwd+bwd, "
                       f"one process per core ({cores} workers: the host's CPU share for one GPU; {affinity} "
                       f"cores in the affinity mask); tokens/s counts all {case.H} heads ({wall:.1f} s)")}


def bench_cw(a):
    """The channel-wise path (per-channel g, b, w) on B4 T4096 H16 d128: one JSON line."""
    import time

    import numpy as np
    import torch

    import workloads as W
    from paper_2608_12700_amd import gdn

    B, T, H, dk, dv = 4, 4096, 16, 128, 128
    bf = a.cw_io == "bf16"
    case = W.make_cw_case("cw_B4_T4096_H16_d128", B, T, H, dk, dv, gates="gbw", seed=6, io_dtype=a.cw_io)
    cpu = None if a.no_cpu_baseline else cw_cpu_baseline(case, a.cpu_budget)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t = {n: (None if getattr(case, n) is None else torch.from_numpy(getattr(case, n)).to(dev))
         for n in ("q", "k", "v", "g", "b", "w", "S0", "dO", "dS_T")}
    if bf:
        for n in ("q", "k", "v", "dO"):
            t[n] = t[n].to(torch.bfloat16)
    p = gdn.make_problem(B, T, H, dk, dv, io_dtype=gdn.GDN_BF16 if bf else gdn.GDN_F32)
    nch = gdn.gdn_num_chunks(p)
    o = torch.empty_like(t["v"])
    S_T = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev)
    states = torch.empty((nch, H, dk, dv), dtype=torch.float32, device=dev)
    grads = [torch.empty_like(t[n]) for n in ("q", "k", "v", "g", "b", "w", "S0")]
    wsf = torch.empty(gdn.gdn_cw_fwd_workspace_size(p), dtype=torch.uint8, device=dev)
    wsb = torch.empty(gdn.gdn_cw_bwd_workspace_size(p), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda x: ctypes.c_void_p(x.data_ptr())
    hip = Hip()
    ns = gdn.NUM_STAGES + 1

    def step(evf=None, evb=None):
        rc = gdn.gdn_cw_fwd_ex(p, P(t["q"]), P(t["k"]), P(t["v"]), P(t["g"]), P(t["b"]), P(t["w"]), P(t["S0"]),
                               P(o), P(S_T), P(states), P(wsf), wsf.numel(), ctypes.c_void_p(stream), evf)
        assert rc == 0, rc
        rc = gdn.gdn_cw_bwd_ex(p, P(t["q"]), P(t["k"]), P(t["v"]), P(t["g"]), P(t["b"]), P(t["w"]), P(states),
                               P(t["dO"]), P(t["dS_T"]), *[P(x) for x in grads], P(wsb), wsb.numel(),
                               ctypes.c_void_p(stream), evb)
        assert rc == 0, rc

    for _ in range(a.warmup):
        step()
    flush = torch.empty(512 * 1024 * 1024 // 4, dtype=torch.float32, device=dev)
    evs = [((ctypes.c_void_p * ns)(*[hip.event() for _ in range(ns)]),
            (ctypes.c_void_p * ns)(*[hip.event() for _ in range(ns)])) for _ in range(a.steps)]
    torch.cuda.synchronize()
    for i in range(a.steps):
        flush.fill_(float(i))
        step(*evs[i])
    torch.cuda.synchronize()
    ms_step = sum(hip.ms(ef[0], eb[ns - 1]) for ef, eb in evs) / a.steps
    fwd_names = ("cw_fwd_prep", "cw_fwd_scan", "cw_fwd_exact", None)
    stage_ms = {}
    for ef, eb in evs:
        for j in range(gdn.NUM_STAGES):
            for nm, e in ((fwd_names[j], ef), (gdn.CW_BWD_STAGES[j], eb)):
                if nm is not None:
                    stage_ms[nm] = stage_ms.get(nm, 0.0) + hip.ms(e[j], e[j + 1]) / a.steps
    ok = all(bool(torch.isfinite(x).all()) for x in [o, S_T] + grads)
    km = cw_kernel_model(B, T, H, dk, dv, es=2 if bf else 4)
    dom = max(km, key=lambda n: stage_ms[n])
    dom_s = stage_ms[dom] / 1e3
    ach = km[dom][0] / dom_s / 1e9
    res = {
        "metric": f"GDN channel-wise (per-channel g, b, w) fwd+bwd tokens/s at B4 T4096 H16 d128 {a.cw_io}",
        "value": round(B * T / (ms_step / 1e3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": ("bf16+f32 (bf16 activations; scans and value-part gradients on bf16 matrix cores, "
                                             "prep and channel gradients in f32)" if bf else "f32"),
        "data": "synthetic (seeded: q,k L2-normalised N(0,1); v,dO N(0,1); g=-softplus(N) per channel; "
                "b=sigmoid(N) per channel; w=1.5*sigmoid(N) per channel; S0 N(0,0.1^2); dS_T N(0,1))",
        "config": {"workload": f"channel-wise gated delta rule fwd+bwd (full GDN gates), {a.cw_io} activations, "
                               "fp32 gates, state and operands, B=4 T=4096 H=16 dk=dv=128 chunk=64",
                   "B": B, "T": T, "H": H, "dk": dk, "dv": dv, "io": a.cw_io},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(dom, CW_TRAFFIC_FILE),
                     "algorithmic_bytes_per_launch": int(km[dom][0]), "avg_launch_ms": round(stage_ms[dom], 4),
                     "mfma_tflops": round(km[dom][1] / dom_s / 1e12, 1)},
        "timing": {"cold_caches": True, "note": "mean of per-step HIP event intervals, each step after a "
                                                "512 MiB scratch write"},
        "path": {"stage_ms": {k_: round(x, 4) for k_, x in stage_ms.items()}, "outputs_finite": ok},
    }
    if a.stages:
        for nm, x in stage_ms.items():
            if nm not in km:  # the exact pass (reads its flags; recomputes flagged streams only)
                print(f"{nm:14s} {x*1e3:9.1f} us", file=sys.stderr)
                continue
            b_, f_ = km[nm]
            print(f"{nm:14s} {x*1e3:9.1f} us  {b_/(x/1e3)/1e9:8.1f} GB/s  {f_/(x/1e3)/1e12:7.1f} TFLOP/s",
                  file=sys.stderr)
    if cpu is not None:
        res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)
    return 0


def path_model(B, T, H, dk, dv, es, N=None, nch=None):
    """The API's compulsory bytes for the forward and the backward (nch: the
    number of chunk states, sum over sequences of ceil(L_n / 64))."""
    N = B if N is None else N
    tok = B * T * H
    nch = B * (-(-T // CH)) if nch is None else nch
    states = nch * H * dk * dv * 4
    s = N * H * dk * dv * 4
    fwd = tok * (2 * dk * es + dv * es + 8) + s + tok * dv * es + s + states
    bwd = tok * (2 * dk * es + dv * es + 8) + states + tok * dv * es + s + tok * (2 * dk * es + dv * es + 8) + s
    return fwd, bwd


class Hip:
    """The few HIP runtime calls the timing needs (events on the launch stream)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        assert self.lib.hipEventCreate(ctypes.byref(e)) == 0
        return e

    def record(self, e, stream):
        assert self.lib.hipEventRecord(e, ctypes.c_void_p(stream)) == 0

    def ms(self, a, b):
        x = ctypes.c_float()
        assert self.lib.hipEventElapsedTime(ctypes.byref(x), a, b) == 0
        return float(x.value)


def host_workers():
    """(workers, cores in the affinity mask): one worker per core, at most 16 (the
    CPU share of one GPU on the measurement hosts)."""
    aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(aff, 16)), aff


def _oracle_stream(args):
    """One (b, h) stream through the float64 oracle: forward then backward."""
    os.environ["OMP_NUM_THREADS"] = os.environ["OPENBLAS_NUM_THREADS"] = "1"
    os.environ["MKL_NUM_THREADS"] = "1"
    import numpy as np
    from oracle import gdn_oracle as O
    q, k, v, g, b, S0, dO, dST = args
    f = lambda x: x[None].astype(np.float64)
    O.fwd_streams(f(q), f(k), f(v), f(g), f(b), f(S0))
    O.bwd_streams(f(q), f(k), f(v), f(g), f(b), f(S0), f(dO), f(dST))
    return q.shape[0]


def cpu_baseline(case, budget_s=15.0):
    """Time the oracle on a bounded sample of the workload's streams, all host cores."""
    import multiprocessing as mp
    cores, affinity = host_workers()
    streams = [(b, h) for b in range(case.B) for h in range(case.H)]
    per_stream_s = 2.5 * (case.T / 4096) * (case.dk * case.dv / 16384)
    n = int(max(cores, min(len(streams), budget_s * cores / max(per_stream_s, 1e-3))))
    n = min(n, len(streams))
    sample = streams[:n]
    tasks = [(case.q[b, :, h], case.k[b, :, h], case.v[b, :, h], case.g[b, :, h], case.beta[b, :, h],
              case.S0[b, h], case.dO[b, :, h], case.dS_T[b, h]) for (b, h) in sample]
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        done = sum(pool.map(_oracle_stream, tasks, chunksize=1))
    wall = time.perf_counter() - t0
    token_heads = done
    return {
        "value": round(token_heads / case.H / wall, 1),
        "unit": "tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"{n} of {len(streams)} (b,h) streams of the workload, full T={case.T} each, "
                   f"float64 token-serial fwd+bwd, one process per core ({cores} workers: the "
                   f"host's CPU share for one GPU; {affinity} cores in the affinity mask); tokens/s "
                   f"counts all {case.H} heads ({token_heads} token-heads in {wall:.1f} s)"),
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--stages", action="store_true", help="also print per-stage timings to stderr")
    ap.add_argument("--copy-kernel", action="store_true",
                    help="only run a plain device copy (calibrates the HBM byte counters)")
    ap.add_argument("--summarize-counters", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="write the traffic summary from four rocprofv3 --pmc output folders")
    ap.add_argument("--summarize-trace", metavar="TRACE", help="write the kernel-trace summary of a "
                    "rocprofv3 --kernel-trace --stats --output-format csv folder")
    ap.add_argument("--summarize-sq", nargs="+", metavar="DIR", help="write the SQ counter summary of "
                    "rocprofv3 --pmc output folders (one per pass)")
    ap.add_argument("--command", default="", help="the profiling command recorded in the summary")
    ap.add_argument("--cw", action="store_true",
                    help="measure the channel-wise path (per-channel g, b, w) instead")
    ap.add_argument("--cw-io", choices=("bf16", "f32"), default="bf16",
                    help="activation dtype of the channel-wise measurement")
    ap.add_argument("--workload", choices=("throughput", "long", "varlen"), default="throughput",
                    help="throughput: the metric workload (B4 T4096 H16 d128); long: B1 T65536 H16 d128 "
                         "(1024-chunk reverse scan); varlen: 16 packed sequences, T=32768, dk=128, dv=256")
    ap.add_argument("--long-T", type=int, default=65536, help="T of the long workload")
    ap.add_argument("--trace-out", default="kernel_trace_bf16_B4_T4096_H16_d128.md",
                    help="file name under profiles/ for --summarize-trace")
    a = ap.parse_args(argv)
    if a.copy_kernel:
        copy_kernel()
        return 0
    if a.summarize_trace:
        md = summarize_trace(a.summarize_trace, a.command, *(
            [f"channel-wise gated delta rule fwd+bwd (per-channel g, b, w), {a.cw_io} activations, "
             "B=4 T=4096 H=16 dk=dv=128"] if a.cw else []))
        with open(os.path.join(ROOT, "profiles", a.trace_out), "w") as fh:
            fh.write(md)
        print(md)
        return 0
    if a.summarize_sq:
        t = summarize_sq(a.summarize_sq, a.command)
        with open(SQ_FILE, "w") as fh:
            json.dump(t, fh, indent=1)
        print(json.dumps(t)[:2000])
        return 0
    if a.summarize_counters:
        t = summarize_counters(*a.summarize_counters, a.command, cw=a.cw, cw_es=2 if a.cw_io == "bf16" else 4)
        with open(CW_TRAFFIC_FILE if a.cw else TRAFFIC_FILE, "w") as fh:
            json.dump(t, fh, indent=1)
        print(json.dumps(t))
        return 0
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {a.gpus}); the path shards over "
              f"(sequence, head) streams with no communication, so N GPUs run N independent copies.",
              file=sys.stderr)
        return 2
    if a.cw:
        return bench_cw(a)

    import numpy as np
    import torch

    import workloads as W
    from paper_2608_12700_amd import gdn

    if a.workload == "long":
        case = W.config2(a.long_T)
    elif a.workload == "varlen":
        case = W.config4()
    else:
        case = W.config1()
    # the oracle's worker processes are forked before anything touches the GPU
    # (the CPU baseline is the metric workload's; other workloads are secondary lines)
    cpu = None if (a.no_cpu_baseline or a.workload != "throughput") else cpu_baseline(case, a.cpu_budget)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, T, H, dk, dv = case.B, case.T, case.H, case.dk, case.dv
    bf = torch.bfloat16
    act = lambda x: torch.from_numpy(x).to(dev).to(bf).contiguous()
    f32 = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    q, k, v, dO = act(case.q), act(case.k), act(case.v), act(case.dO)
    g, beta, S0, dST = f32(case.g), f32(case.beta), f32(case.S0), f32(case.dS_T)

    packed = None if case.cu_seqlens is None else gdn.Packed(case.cu_seqlens, dev)
    p = (gdn.make_problem(B, T, H, dk, dv, io_dtype=gdn.GDN_BF16, variant="gated_delta") if packed is None else
         gdn.make_problem(B, T, H, dk, dv, io_dtype=gdn.GDN_BF16, variant="gated_delta", cu_host=packed.host,
                          cu_dev_ptr=packed.dev.data_ptr()))
    nch = gdn.gdn_num_chunks(p)
    N = case.N
    o = torch.empty_like(v)
    S_T = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    states = torch.empty((nch, H, dk, dv), dtype=torch.float32, device=dev)
    dq, dk_, dv_ = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    dg, db = torch.empty_like(g), torch.empty_like(beta)
    dS0 = torch.empty_like(S0)
    wsf = torch.empty(gdn.gdn_fwd_workspace_size(p), dtype=torch.uint8, device=dev)
    wsb = torch.empty(gdn.gdn_bwd_workspace_size(p), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    hip = Hip()
    ns = gdn.NUM_STAGES + 1

    def step(evf=None, evb=None):
        rc = gdn.gdn_fwd_ex(p, P(q), P(k), P(v), P(g), P(beta), P(S0), P(o), P(S_T), P(states), P(wsf),
                            wsf.numel(), ctypes.c_void_p(stream), evf)
        assert rc == 0, rc
        rc = gdn.gdn_bwd_ex(p, P(q), P(k), P(v), P(g), P(beta), P(states), P(dO), P(dST), P(dq), P(dk_),
                            P(dv_), P(dg), P(db), P(dS0), P(wsb), wsb.numel(), ctypes.c_void_p(stream), evb)
        assert rc == 0, rc

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # Timed region 1: K steps back to back, bracketed by synchronisations.
    t0, t1 = hip.event(), hip.event()
    torch.cuda.synchronize()
    hip.record(t0, stream)
    for _ in range(a.steps):
        step()
    hip.record(t1, stream)
    torch.cuda.synchronize()
    ms_step_warm = hip.ms(t0, t1) / a.steps

    # Timed region 2 (the reported figure): every step starts with cold caches --
    # a 512 MiB scratch write evicts L2 and the 256 MB MALL, which could otherwise
    # hold the 268 MB of chunk states between the forward and the backward of the
    # previous step -- and is timed alone with HIP events on the launch stream
    # (stage boundaries included), so the flush itself is never timed.
    flush = torch.empty(512 * 1024 * 1024 // 4, dtype=torch.float32, device=dev)
    evs = []
    for _ in range(a.steps):
        ef = (ctypes.c_void_p * ns)(*[hip.event() for _ in range(ns)])
        eb = (ctypes.c_void_p * ns)(*[hip.event() for _ in range(ns)])
        evs.append((ef, eb))
    torch.cuda.synchronize()
    for i in range(a.steps):
        flush.fill_(float(i))
        step(evs[i][0], evs[i][1])
    torch.cuda.synchronize()
    per_step = sorted(hip.ms(ef[0], eb[ns - 1]) for ef, eb in evs)
    ms_step = sum(per_step) / a.steps
    q_ = lambda f: per_step[min(len(per_step) - 1, int(f * (len(per_step) - 1) + 0.5))]
    del flush

    names = list(gdn.FWD_STAGES) + list(gdn.BWD_STAGES)
    stage_ms = {nm: 0.0 for nm in names}
    for ef, eb in evs:
        for j in range(gdn.NUM_STAGES):
            stage_ms[gdn.FWD_STAGES[j]] += hip.ms(ef[j], ef[j + 1]) / a.steps
            stage_ms[gdn.BWD_STAGES[j]] += hip.ms(eb[j], eb[j + 1]) / a.steps
    stage_ms.pop(None, None)  # a direction with fewer stages leaves the last one empty
    names = [n for n in names if n is not None]
    fwd_ms = sum(stage_ms[n] for n in gdn.FWD_STAGES if n is not None)
    bwd_ms = sum(stage_ms[n] for n in gdn.BWD_STAGES if n is not None)

    ok = all(bool(torch.isfinite(x).all()) for x in (o, S_T, dq, dk_, dv_, dg, db, dS0))

    km = kernel_model(B, T, H, dk, dv, 2, N=N, nch=nch)
    dom = max(km, key=lambda n: stage_ms[n])
    dom_bytes, dom_flops = km[dom]
    dom_s = stage_ms[dom] / 1e3
    fwd_b, bwd_b = path_model(B, T, H, dk, dv, 2, N=N, nch=nch)
    main = a.workload == "throughput"
    traffic = measured_traffic if main else (lambda st: None)  # counters were taken on the metric workload
    # the backward against its compulsory API bytes (each tensor of the gdn_bwd
    # call read or written once at its dtype; workspace traffic excluded)
    bwd_s = bwd_ms / 1e3
    ach = bwd_b / bwd_s / 1e9
    state_io = 2 * N * H * dk * dv * 4  # dS_T in, dS0 out: moved by the reverse scan
    grad_api = bwd_b - state_io         # everything else passes through the gradient kernel
    bwd_traffic = [traffic(st) for st in ("bwd_prep", "bwd_scan", "bwd_grad")]

    tokens = B * T
    res = {
        "metric": "GDN fwd+bwd tokens/s at B4 T4096 H16 d128 bf16; % of binding roofline",
        "value": round(tokens / (ms_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded: q,k L2-normalised N(0,1); v,dO N(0,1); beta=sigmoid(N); "
                "g=-0.1*softplus(N); S0 N(0,0.1^2); dS_T N(0,1))",
        "config": {"workload": "gated delta rule fwd+bwd, bf16 I/O, fp32 state, B=4 T=4096 H=16 "
                               "dk=dv=128 chunk=64", "B": B, "T": T, "H": H, "dk": dk, "dv": dv,
                   "chunk": CH, "global_batch": B, "seq_len": T, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": "gdn_bwd (bwd_prep + bwd_scan + bwd_grad + bwd_exact)",
                     "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBS, 4),
                     "traffic": (sum(bwd_traffic) if all(x is not None for x in bwd_traffic) else None),
                     "algorithmic_bytes_per_launch": int(bwd_b),
                     "avg_launch_ms": round(bwd_ms, 4),
                     "stage_ms": {n: round(stage_ms[n], 4) for n in gdn.BWD_STAGES},
                     "dominant_kernel": {
                         "kernel": dom, "avg_launch_ms": round(stage_ms[dom], 4),
                         "compulsory_bytes": int(grad_api),
                         "achieved": round(grad_api / dom_s / 1e9, 1),
                         "frac": round(grad_api / dom_s / 1e9 / HBM_PEAK_GBS, 4),
                         "kernel_io_bytes": int(dom_bytes),
                         "kernel_io_frac": round(dom_bytes / dom_s / 1e9 / HBM_PEAK_GBS, 4),
                         "traffic": traffic(dom),
                         "mfma_tflops": round(dom_flops / dom_s / 1e12, 1)}},
        "timing": {"cold_caches": True, "median_ms": round(q_(0.5), 4),
                   "iqr_ms": [round(q_(0.25), 4), round(q_(0.75), 4)],
                   "back_to_back_ms_per_step": round(ms_step_warm, 4),
                   "back_to_back_tokens_per_s": round(tokens / (ms_step_warm / 1e3), 1),
                   "note": "value and ms_per_step: mean of per-step HIP event intervals, each step "
                           "after a 512 MiB scratch write (L2 and MALL cold); back_to_back: the same "
                           "K steps bracketed as one region without flushes"},
        "path": {"fwd_ms": round(fwd_ms, 4), "bwd_ms": round(bwd_ms, 4),
                 "fwd_hbm_frac": round(fwd_b / 8e12 / (fwd_ms / 1e3), 4),
                 "bwd_hbm_frac": round(bwd_b / 8e12 / (bwd_ms / 1e3), 4),
                 "bwd_tokens_per_s": round(tokens / (bwd_ms / 1e3), 1),
                 "stage_ms": {k_: round(x, 4) for k_, x in stage_ms.items()},
                 "outputs_finite": ok},
    }
    # the reverse scan's serial chain: time per chunk step of the longest stream
    max_nch = max(-(-L // CH) for (_, _, L) in case.seq_bounds())
    res["path"]["chunks_per_stream"] = max_nch
    res["path"]["fwd_scan_us_per_chunk"] = round(stage_ms["fwd_scan"] * 1e3 / max_nch, 3)
    res["path"]["bwd_scan_us_per_chunk"] = round(stage_ms["bwd_scan"] * 1e3 / max_nch, 3)
    if not main:
        # a secondary line: the same measurement on another specified workload
        what = {"long": f"B1 T{T} H16 d128 bf16 (long-sequence reverse-state stress, g=-0.02*softplus(N))",
                "varlen": "packed varlen 16 sequences T32768 H16 dk128 dv256 bf16"}[a.workload]
        res["metric"] = f"GDN fwd+bwd tokens/s at {what}; % of binding roofline"
        res["data"] = res["data"].replace("g=-0.1", "g=-0.02") if a.workload == "long" else res["data"]
        res["config"] = {"workload": f"gated delta rule fwd+bwd, {what}, chunk=64", "B": B, "T": T, "H": H,
                         "dk": dk, "dv": dv, "chunk": CH, "num_seqs": N, "chunk_states": nch,
                         "parallelism": "none (1 GPU)"}
        if a.workload == "varlen":
            res["config"]["cu_seqlens"] = [int(x) for x in case.cu_seqlens]
    if a.stages:
        for nm in names:
            b_, f_ = km.get(nm, (0, 0))
            t_ = stage_ms[nm] / 1e3
            if t_ > 0 and b_:
                print(f"{nm:10s} {stage_ms[nm]*1e3:9.1f} us  {b_/t_/1e9:8.1f} GB/s  {f_/t_/1e12:7.1f} TFLOP/s",
                      file=sys.stderr)
    if cpu is not None:
        res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

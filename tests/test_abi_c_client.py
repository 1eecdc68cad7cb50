"""The C interface from a C program: tests/abi_client.c, compiled with gcc as
C99 against include/gdn.h and linked to libgdn.so, with no Python in its path.

* CPU: the header compiles as C with -Wall -Wextra -Werror, and the client's
  host-side checks pass (chunk counts, workspace sizes, the status codes of
  malformed calls), without a GPU.
* GPU: the client reads seeded inputs from a file, allocates device memory
  with hipMalloc, runs gdn_fwd and gdn_bwd on the default stream and writes
  every output back; the outputs must match the float64 oracle to the dtype's
  tolerance.  The client is started from a worker process that was forked
  before this process touched the GPU.
"""
import os
import subprocess

import numpy as np
import pytest

import workloads as W
from tests import harness as Hn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
MAGIC = 0x31444E47
VARIANT = {"gated_delta": 0, "delta": 1, "decay_only": 2}


def _build(out_dir):
    exe = os.path.join(out_dir, "abi_client")
    lib = os.path.join(ROOT, "paper_2608_12700_amd")
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           os.path.join(ROOT, "tests", "abi_client.c"), "-o", exe,
           "-L", lib, "-lgdn", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{lib}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    return exe


def _run_client(args):
    """Runs in an oracle-pool worker (no GPU context in that process)."""
    r = subprocess.run(list(args), capture_output=True, text=True, timeout=120)
    return r.returncode, r.stdout, r.stderr


def test_c_client_host_checks(tmp_path):
    exe = _build(str(tmp_path))
    r = subprocess.run([exe, "host"], capture_output=True, text=True, timeout=60)
    print(r.stdout, r.stderr)
    assert r.returncode == 0 and "host checks passed" in r.stdout, (r.returncode, r.stdout, r.stderr)


def _bits(x, io):
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16) if io == "bf16" else x


def _write_inputs(path, c, has_S0, has_dST):
    packed = c.cu_seqlens is not None
    hd = [MAGIC, c.B, c.T, c.H, c.dk, c.dv, 1 if c.io_dtype == "bf16" else 0, VARIANT[c.variant], c.N,
          int(packed), int(has_S0), int(has_dST)]
    with open(path, "wb") as f:
        f.write(np.asarray(hd, dtype=np.int32).tobytes())
        if packed:
            f.write(np.asarray(c.cu_seqlens, dtype=np.int32).tobytes())
        for x in (c.q, c.k, c.v):
            f.write(_bits(x, c.io_dtype).tobytes())
        for x in (c.g, c.beta):
            if x is not None:
                f.write(np.ascontiguousarray(x, dtype=np.float32).tobytes())
        if has_S0:
            f.write(np.ascontiguousarray(c.S0, dtype=np.float32).tobytes())
        f.write(_bits(c.dO, c.io_dtype).tobytes())
        if has_dST:
            f.write(np.ascontiguousarray(c.dS_T, dtype=np.float32).tobytes())


def _read_outputs(path, c, nch):
    raw = open(path, "rb").read()
    off = 0
    bf = c.io_dtype == "bf16"

    def take(shape, act):
        nonlocal off
        n = int(np.prod(shape))
        if act and bf:
            u = np.frombuffer(raw, np.uint16, n, off).astype(np.uint32) << 16
            off += 2 * n
            return u.view(np.float32).reshape(shape).astype(np.float64)
        x = np.frombuffer(raw, np.float32, n, off).reshape(shape).astype(np.float64)
        off += 4 * n
        return x

    B, T, H, dk, dv, N = c.B, c.T, c.H, c.dk, c.dv, c.N
    out = dict(o=take((B, T, H, dv), True), S_T=take((N, H, dk, dv), False),
               states=take((nch, H, dk, dv), False), dq=take((B, T, H, dk), True),
               dk=take((B, T, H, dk), True), dv=take((B, T, H, dv), True))
    out["dg"] = take((B, T, H), False) if c.g is not None else None
    out["dbeta"] = take((B, T, H), False) if c.beta is not None else None
    out["dS0"] = take((N, H, dk, dv), False)
    assert off == len(raw), (off, len(raw))
    return out


CASES = {
    "bf16_gated_B2_T130_d128": lambda: (W.make_case("c_client_bf16", B=2, T=130, H=2, dk=128, dv=128, seed=51),
                                        True, True),
    "f32_delta_packed_d64x128": lambda: (W.make_case("c_client_f32_packed", B=1, T=200, H=2, dk=64, dv=128,
                                                     io_dtype="f32", variant="delta", seed=52,
                                                     cu_seqlens=np.array([0, 5, 70, 70, 200], np.int32)),
                                         False, False),
    "bf16_decay_B1_T100_d128x64": lambda: (W.make_case("c_client_bf16_decay", B=1, T=100, H=3, dk=128, dv=64,
                                                       variant="decay_only", decay_scale=1.0, seed=53),
                                           True, False),
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
def test_c_client_matches_oracle(tmp_path, name):
    from tests import oracle_pool
    if oracle_pool._POOL is None:
        pytest.skip("needs the worker pool forked before this process used the GPU")
    c, has_S0, has_dST = CASES[name]()
    if not has_S0:
        c.S0[...] = 0.0  # the client passes NULL: the oracle starts from zero
    if not has_dST:
        c.dS_T[...] = 0.0
    exe = _build(str(tmp_path))
    inp, out = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    _write_inputs(inp, c, has_S0, has_dST)
    print("case", W.describe(c), "S0" if has_S0 else "no S0", "dS_T" if has_dST else "no dS_T", flush=True)
    rc, so, se = oracle_pool.pool().apply(_run_client, ((exe, "run", inp, out),))
    print(so, se, flush=True)
    assert rc == 0, (rc, so, se)
    nch = sum(-(-L // 64) for _, _, L in c.seq_bounds())
    dev = _read_outputs(out, c, nch)
    ref = Hn.run_oracle(c)
    res = Hn.compare(dev, ref)
    print({k: (f"{v[0]:.2e}", v[1]) for k, v in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL[c.io_dtype], name)

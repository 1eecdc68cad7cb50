"""Channel-wise members on the GPU against the float64 channel-wise oracle.

Every case calls the C ABI (gdn_cw_fwd / gdn_cw_bwd through the binding) on
seeded inputs and compares every output with the oracle at the bar of its
activation dtype (rel-L2 <= 1e-4 per tensor for fp32, 1e-2 for bf16; the
oracle sees the same once-rounded values):

* full GDN gates (per-channel g, b, w), KDA (b = w = beta broadcast), GLA
  (g only), LA (no gates), each over several chunks and a ragged tail;
* bf16 activations for every member and for packed sequences; empty
  sequences (inside a packed batch, and T = 0);
* d_k / d_v in {64, 128, 256} combinations, packed variable-length
  sequences (including a one-token sequence), a T shorter than one chunk;
* a strong decay (mean log-decay about -4 per token and channel, tails near
  -15): the chunked kernels split every decay so that no factor exceeds 1;
  and strong and weak 16-token blocks mixed inside each chunk (exact and
  matrix-core in-block sums side by side);
* the throughput shape (B4 T4096 H16 d128) in the launch configuration the
  bench times, checked on sampled heads;
* run-to-run bitwise determinism, and fwd + bwd captured in a HIP graph with
  every replay bitwise equal to eager execution.
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
    return None if x is None else x.detach().float().cpu().numpy().astype(np.float64)


def run_device(c: W.CwCase):
    from paper_2608_12700_amd import gdn
    t = {n: _dev(getattr(c, n)) for n in ("q", "k", "v", "g", "b", "w", "S0", "dO", "dS_T")}
    if c.io_dtype == "bf16":  # the arrays hold bf16 values already: the cast is exact
        for n in ("q", "k", "v", "dO"):
            t[n] = t[n].to(torch.bfloat16)
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
    Hn.assert_parity(res, Hn.TOL[c.io_dtype], c.name)
    return dev


@pytest.mark.parametrize("gates", ["gbw", "kda", "g", ""])
def test_members_small(gates):
    check(W.make_cw_case(f"cw_{gates or 'la'}", 2, 200, 2, 64, 64, gates=gates, seed=1))


@pytest.mark.parametrize("dk,dv", [(128, 128), (128, 64), (64, 256), (128, 256)])
def test_dims_full_gates(dk, dv):
    check(W.make_cw_case(f"cw_d{dk}_{dv}", 1, 131, 2, dk, dv, gates="gbw", seed=2))


@pytest.mark.parametrize("gates", ["gbw", "kda", "g", ""])
def test_members_bf16_io(gates):
    check(W.make_cw_case(f"cw_bf16_{gates or 'la'}", 2, 200, 2, 128, 128, gates=gates, seed=12, io_dtype="bf16"))


def test_packed_sequences_bf16_io():
    cu = np.array([0, 1, 65, 200, 331], dtype=np.int32)
    check(W.make_cw_case("cw_packed_bf16", 1, 331, 2, 64, 256, gates="gbw", seed=13, cu_seqlens=cu,
                         io_dtype="bf16"))


def test_packed_sequences():
    cu = np.array([0, 70, 71, 200, 333], dtype=np.int32)
    check(W.make_cw_case("cw_packed", 1, 333, 2, 128, 128, gates="gbw", seed=3, cu_seqlens=cu))


def test_empty_sequences():
    # an empty sequence inside a packed batch carries S0 to S_T and dS_T to dS0;
    # T = 0 overall leaves nothing but the states
    cu = np.array([0, 70, 70, 71, 200], dtype=np.int32)
    check(W.make_cw_case("cw_packed_empty", 1, 200, 2, 64, 128, gates="gbw", seed=14, cu_seqlens=cu))
    check(W.make_cw_case("cw_T0", 2, 0, 2, 64, 64, gates="kda", seed=15))


def test_shorter_than_one_chunk():
    check(W.make_cw_case("cw_short", 3, 17, 1, 64, 128, gates="kda", seed=4))


def test_strong_decay():
    # a 16-token block decays by ~65 on average and by far more in the tails:
    # a single reference per block would overflow fp32 here
    check(W.make_cw_case("cw_strong", 1, 192, 2, 128, 128, gates="gbw", seed=5, decay=5.0))


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_mixed_decay_blocks(io):
    # every third 16-token block decays strongly (its in-block pairs are summed
    # exactly), the others weakly (they go to the matrix cores), inside the
    # same chunks; the ragged tail ends in a strong block
    T = 200
    scale = np.where((np.arange(T) // 16) % 3 == 0, 8.0, 0.3)
    check(W.make_cw_case(f"cw_mixed_{io}", 2, T, 2, 128, 128, gates="gbw", seed=16, decay=scale, io_dtype=io))


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_throughput_shape_sampled_heads(io):
    c = W.make_cw_case("cw_B4_T4096_H16_d128", 4, 4096, 16, 128, 128, gates="gbw", seed=6, io_dtype=io)
    check(c, heads=[0, 11])


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_deterministic_bitwise(io):
    c = W.make_cw_case(f"cw_det_{io}", 1, 300, 3, 128, 128, gates="gbw", seed=7, io_dtype=io)
    a, b = run_device(c), run_device(c)
    for n in NAMES:
        if a[n] is not None:
            assert np.array_equal(a[n], b[n], equal_nan=True), n


def test_graph_capture_replay_bitwise():
    """gdn_cw_fwd + gdn_cw_bwd recorded once into a HIP graph and replayed with eager
    work and synchronisations between replays; every replay equals eager bit for bit."""
    import ctypes
    from paper_2608_12700_amd import gdn
    c = W.make_cw_case("cw_graph", 2, 200, 3, 128, 128, gates="gbw", seed=8)
    t = {n: _dev(getattr(c, n)) for n in ("q", "k", "v", "g", "b", "w", "S0", "dO", "dS_T")}
    dev = t["q"].device
    p = gdn.make_problem(c.B, c.T, c.H, c.dk, c.dv, io_dtype=gdn.GDN_F32)
    nch = gdn.gdn_num_chunks(p)
    outs = dict(o=torch.empty_like(t["v"]),
                S_T=torch.empty((c.B, c.H, c.dk, c.dv), dtype=torch.float32, device=dev),
                states=torch.empty((nch, c.H, c.dk, c.dv), dtype=torch.float32, device=dev))
    for n in ("q", "k", "v", "g", "b", "w", "S0"):
        outs["d" + n] = torch.empty_like(t[n])
    wsf = torch.empty(gdn.gdn_cw_fwd_workspace_size(p), dtype=torch.uint8, device=dev)
    wsb = torch.empty(gdn.gdn_cw_bwd_workspace_size(p), dtype=torch.uint8, device=dev)
    P = lambda x: ctypes.c_void_p(x.data_ptr())

    def step():
        s = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        assert gdn.gdn_cw_fwd(p, P(t["q"]), P(t["k"]), P(t["v"]), P(t["g"]), P(t["b"]), P(t["w"]), P(t["S0"]),
                              P(outs["o"]), P(outs["S_T"]), P(outs["states"]), P(wsf), wsf.numel(), s) == 0
        assert gdn.gdn_cw_bwd(p, P(t["q"]), P(t["k"]), P(t["v"]), P(t["g"]), P(t["b"]), P(t["w"]),
                              P(outs["states"]), P(t["dO"]), P(t["dS_T"]), P(outs["dq"]), P(outs["dk"]),
                              P(outs["dv"]), P(outs["dg"]), P(outs["db"]), P(outs["dw"]), P(outs["dS0"]), P(wsb),
                              wsb.numel(), s) == 0

    step()
    torch.cuda.synchronize()
    eager = {n: x.clone() for n, x in outs.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        for x in outs.values():
            x.fill_(float("nan"))
        wsf.fill_(rep + 1)
        wsb.fill_(rep + 2)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n, x in outs.items():
            assert torch.equal(x.view(torch.uint8), eager[n].view(torch.uint8)), (rep, n)
        step()
        torch.cuda.synchronize()
        for n, x in outs.items():
            assert torch.equal(x.view(torch.uint8), eager[n].view(torch.uint8)), ("eager", rep, n)

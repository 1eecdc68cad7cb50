"""Tensors past 2^31 elements: every element offset of the path is 64-bit.

Fixed-length layout: B = 8448 sequences of T = 1000 tokens (each ends in a ragged 40-token chunk),
H = 2, d_k = d_v = 128, bf16: q, k, v, dO, o and their gradients hold 2.16e9
elements each (4.3 GB), so the last sequences start past element 2^31, and the
chunk states (17.7 GB) and both workspaces (20 and 27 GB) are far past 2^31
bytes.  Three sequences -- the first and the last two -- carry seeded inputs
of the case generator and are compared with the float64 oracle to the bf16
tolerance; the rest of the batch is filled on the device with seeded random
values of the same distributions, and every output of every sequence must be
finite.  About 105 GB of device memory.

Packed layout: 8500 sequences of seeded lengths 1..1999 in one row
(cu_seqlens), the same sizes, the first and the last two sequences checked
the same way.
"""
import numpy as np
import pytest

import workloads as W
from tests import harness as Hn

pytestmark = pytest.mark.gpu

B, T, H, D = 8448, 1000, 2, 128
ROWS = (0, B - 2, B - 1)  # the sequences checked against the oracle


def _fill(shape, gen, normalize):
    """bf16 activations drawn on the device, a slice along the first axis at a time."""
    import torch
    import torch.nn.functional as F
    x = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    step = max(1, (1 << 28) // int(np.prod(shape[1:])))  # 1 GiB of fp32 draws at a time
    for b0 in range(0, shape[0], step):
        y = torch.randn((min(step, shape[0] - b0),) + tuple(shape[1:]), generator=gen, device="cuda")
        if normalize:
            y = F.normalize(y, dim=-1)
        x[b0:b0 + y.shape[0]] = y.to(torch.bfloat16)
        del y
    return x


def _check(dev, c, label):
    import torch
    torch.cuda.empty_cache()
    ref = Hn.run_oracle(c)
    res = Hn.compare(dev, ref)
    print({k_: (f"{r[0]:.2e}", r[1]) for k_, r in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL["bf16"], label)


def test_offsets_past_2_31():
    import torch
    import torch.nn.functional as F
    from paper_2608_12700_amd import gdn
    assert (B - 2) * T * H * D > 2 ** 31  # the last two sequences start past element 2^31
    torch.cuda.empty_cache()
    print(f"case B={B} T={T} H={H} d={D} bf16 ({B * T * H * D} elements per activation)", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    q, k = _fill((B, T, H, D), gen, True), _fill((B, T, H, D), gen, True)
    v, dO = _fill((B, T, H, D), gen, False), _fill((B, T, H, D), gen, False)
    g = -0.1 * F.softplus(torch.randn((B, T, H), generator=gen, device="cuda"))
    beta = torch.sigmoid(torch.randn((B, T, H), generator=gen, device="cuda"))
    S0 = 0.1 * torch.randn((B, H, D, D), generator=gen, device="cuda")
    dST = torch.randn((B, H, D, D), generator=gen, device="cuda")
    c = W.make_case("large_offsets_rows", B=len(ROWS), T=T, H=H, dk=D, dv=D, seed=29)
    small = Hn.device_inputs(c)
    for i, b in enumerate(ROWS):
        for name, big in (("q", q), ("k", k), ("v", v), ("dO", dO), ("g", g), ("beta", beta),
                          ("S0", S0), ("dS_T", dST)):
            big[b] = small[name][i]
    del small
    torch.cuda.synchronize()
    print("inputs ready", flush=True)

    o, S_T, states = gdn.fwd(q, k, v, g, beta, S0)
    dq, dk, dv, dg, db, dS0 = gdn.bwd(q, k, v, g, beta, states, dO, dST)
    torch.cuda.synchronize()
    print("forward and backward done", flush=True)
    outs = dict(o=o, S_T=S_T, states=states, dq=dq, dk=dk, dv=dv, dg=dg, dbeta=db, dS0=dS0)
    for name, x in outs.items():
        assert bool(torch.isfinite(x).all()), name

    nt = -(-T // 64)
    rows = torch.tensor(ROWS, device="cuda")
    srows = torch.cat([torch.arange(b * nt, (b + 1) * nt, device="cuda") for b in ROWS])
    npy = lambda x: x.float().cpu().numpy().astype(np.float64)
    dev = {name: npy(x.index_select(0, srows if name == "states" else rows)) for name, x in outs.items()}
    del q, k, v, dO, g, beta, S0, dST, outs, o, S_T, states, dq, dk, dv, dg, db, dS0
    _check(dev, c, "large offsets")


def test_packed_offsets_past_2_31():
    import torch
    import torch.nn.functional as F
    from paper_2608_12700_amd import gdn
    N = 8500
    lens = np.random.Generator(np.random.PCG64(31)).integers(1, 2000, size=N)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    Tt = int(cu[-1])
    assert int(cu[N - 2]) * H * D > 2 ** 31 and Tt < 2 ** 31
    nts = -(-lens // 64)
    coff = np.concatenate([[0], np.cumsum(nts)])
    sel = (0, N - 2, N - 1)
    torch.cuda.empty_cache()
    print(f"case packed N={N} T={Tt} H={H} d={D} bf16 ({Tt * H * D} elements per activation)", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    q, k = _fill((Tt, H, D), gen, True), _fill((Tt, H, D), gen, True)
    v, dO = _fill((Tt, H, D), gen, False), _fill((Tt, H, D), gen, False)
    q, k, v, dO = (x.view(1, Tt, H, D) for x in (q, k, v, dO))
    g = -0.1 * F.softplus(torch.randn((1, Tt, H), generator=gen, device="cuda"))
    beta = torch.sigmoid(torch.randn((1, Tt, H), generator=gen, device="cuda"))
    S0 = 0.1 * torch.randn((N, H, D, D), generator=gen, device="cuda")
    dST = torch.randn((N, H, D, D), generator=gen, device="cuda")
    scu = np.concatenate([[0], np.cumsum([lens[n] for n in sel])]).astype(np.int32)
    c = W.make_case("large_offsets_packed_rows", B=1, T=int(scu[-1]), H=H, dk=D, dv=D, seed=37, cu_seqlens=scu)
    small = Hn.device_inputs(c)
    for i, n in enumerate(sel):
        a, b = int(cu[n]), int(cu[n + 1])
        sa, sb = int(scu[i]), int(scu[i + 1])
        for name, big in (("q", q), ("k", k), ("v", v), ("dO", dO), ("g", g), ("beta", beta)):
            big[0, a:b] = small[name][0, sa:sb]
        S0[n] = small["S0"][i]
        dST[n] = small["dS_T"][i]
    del small
    torch.cuda.synchronize()
    print("inputs ready", flush=True)

    packed = gdn.Packed(cu.astype(np.int32), "cuda")
    o, S_T, states = gdn.fwd(q, k, v, g, beta, S0, cu_seqlens=packed)
    dq, dk, dv, dg, db, dS0 = gdn.bwd(q, k, v, g, beta, states, dO, dST, cu_seqlens=packed)
    torch.cuda.synchronize()
    print("forward and backward done", flush=True)
    outs = dict(o=o, S_T=S_T, states=states, dq=dq, dk=dk, dv=dv, dg=dg, dbeta=db, dS0=dS0)
    for name, x in outs.items():
        assert bool(torch.isfinite(x).all()), name

    tok = torch.cat([torch.arange(int(cu[n]), int(cu[n + 1]), device="cuda") for n in sel])
    chk = torch.cat([torch.arange(int(coff[n]), int(coff[n + 1]), device="cuda") for n in sel])
    seqs = torch.tensor(sel, device="cuda")
    npy = lambda x: x.float().cpu().numpy().astype(np.float64)
    dev = {}
    for name, x in outs.items():
        if name in ("S_T", "dS0"):
            dev[name] = npy(x.index_select(0, seqs))
        elif name == "states":
            dev[name] = npy(x.index_select(0, chk))
        else:
            dev[name] = npy(x.index_select(1, tok))
    del q, k, v, dO, g, beta, S0, dST, outs, o, S_T, states, dq, dk, dv, dg, db, dS0
    _check(dev, c, "large offsets, packed")

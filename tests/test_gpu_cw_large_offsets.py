"""Channel-wise members with tensors past 2^31 elements (64-bit element offsets).

B = 8448 sequences of T = 1000 tokens, H = 2, d_k = d_v = 128, bf16
activations with the full per-channel gates: q, k, v, dO, o and their
gradients (bf16) and g, b, w and theirs (fp32) hold 2.16e9 elements each, so
the last sequences start past element 2^31.  The first and the last two
sequences carry seeded inputs of the case generator and are compared with the
float64 channel-wise oracle; the rest is drawn on the device with the same
distributions, and every output must be finite.  About 185 GB of device
memory (the backward's workspace alone is 76 GB).
"""
import numpy as np
import pytest

import workloads as W
from tests import harness as Hn
from tests import test_gpu_cw as TC
from tests.test_gpu_large_offsets import _fill

pytestmark = pytest.mark.gpu

B, T, H, D = 8448, 1000, 2, 128
ROWS = (0, B - 2, B - 1)


def _gate(shape, gen, kind):
    """fp32 per-channel gates drawn on the device, a slice of sequences at a time."""
    import torch
    import torch.nn.functional as F
    x = torch.empty(shape, dtype=torch.float32, device="cuda")
    for b0 in range(0, shape[0], 1024):
        y = torch.randn((min(1024, shape[0] - b0),) + tuple(shape[1:]), generator=gen, device="cuda")
        x[b0:b0 + y.shape[0]] = -F.softplus(y) if kind == "g" else (torch.sigmoid(y) * (1.5 if kind == "w" else 1.0))
        del y
    return x


def test_cw_offsets_past_2_31():
    import torch
    from paper_2608_12700_amd import gdn
    assert (B - 2) * T * H * D > 2 ** 31
    torch.cuda.empty_cache()
    print(f"case channel-wise B={B} T={T} H={H} d={D} bf16 ({B * T * H * D} elements per tensor)", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    q, k = _fill((B, T, H, D), gen, True), _fill((B, T, H, D), gen, True)
    v, dO = _fill((B, T, H, D), gen, False), _fill((B, T, H, D), gen, False)
    g, b, w = (_gate((B, T, H, D), gen, kind) for kind in ("g", "b", "w"))
    S0 = 0.1 * torch.randn((B, H, D, D), generator=gen, device="cuda")
    dST = torch.randn((B, H, D, D), generator=gen, device="cuda")
    c = W.make_cw_case("cw_large_offsets_rows", len(ROWS), T, H, D, D, gates="gbw", seed=41, io_dtype="bf16")
    for i, r in enumerate(ROWS):
        for name, big in (("q", q), ("k", k), ("v", v), ("dO", dO), ("g", g), ("b", b), ("w", w),
                          ("S0", S0), ("dS_T", dST)):
            big[r] = torch.from_numpy(np.ascontiguousarray(getattr(c, name)[i])).to("cuda", big.dtype)
    torch.cuda.synchronize()
    print("inputs ready", flush=True)

    o, S_T, states = gdn.cw_fwd(q, k, v, g, b, w, S0)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()  # the forward's workspace
    grads = gdn.cw_bwd(q, k, v, g, b, w, states, dO, dST)
    torch.cuda.synchronize()
    print("forward and backward done", flush=True)
    outs = dict(o=o, S_T=S_T, states=states, **dict(zip(("dq", "dk", "dv", "dg", "db", "dw", "dS0"), grads)))
    for name, x in outs.items():
        assert bool(torch.isfinite(x).all()), name

    nt = -(-T // 64)
    rows = torch.tensor(ROWS, device="cuda")
    srows = torch.cat([torch.arange(r * nt, (r + 1) * nt, device="cuda") for r in ROWS])
    npy = lambda x: x.float().cpu().numpy().astype(np.float64)
    dev = {name: npy(x.index_select(0, srows if name == "states" else rows)) for name, x in outs.items()}
    del q, k, v, dO, g, b, w, S0, dST, o, S_T, states, grads, outs
    torch.cuda.empty_cache()
    ref = TC.run_oracle(c)
    res = Hn.compare(dev, ref, names=TC.NAMES)
    print({k_: (f"{r_[0]:.2e}", r_[1]) for k_, r_ in res.items()}, flush=True)
    Hn.assert_parity(res, Hn.TOL["bf16"], "channel-wise large offsets")

"""The library used the way a training step uses it.

* autograd: ``gated_delta_rule`` (a torch.autograd.Function over gdn_fwd /
  gdn_bwd) against the float64 oracle, for a loss on both outputs and for a
  loss on ``o`` alone (the backward then sees dS_T = 0);
* graph capture: fwd + bwd recorded once into a HIP graph and replayed several
  times, with eager work and synchronisations between replays; every replay
  must reproduce the eager outputs bit for bit;
* 300-step synthetic training runs at L = 256 (the paper's training length)
  for the gated delta rule and the scalar-decay (SSD) member: a one-layer
  model fitted to a fixed random teacher of the same architecture; the loss
  must fall and stay finite.
"""
import ctypes

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as W
from tests import harness as Hn

pytestmark = pytest.mark.gpu


def _leaf(x):
    return x.detach().clone().requires_grad_(True)


def _np(x):
    return None if x is None else x.detach().float().cpu().numpy().astype(np.float64)


def test_autograd_matches_oracle_fp32():
    from paper_2608_12700_amd.autograd import gated_delta_rule
    case = W.make_case("f32_autograd", B=2, T=130, H=2, dk=64, dv=64, io_dtype="f32")
    print("case", W.describe(case), flush=True)
    t = Hn.device_inputs(case)
    q, k, v, g, beta, S0 = (_leaf(t[n]) for n in ("q", "k", "v", "g", "beta", "S0"))
    o, S_T = gated_delta_rule(q, k, v, g, beta, S0)
    loss = (o * t["dO"]).sum() + (S_T * t["dS_T"]).sum()
    loss.backward()
    torch.cuda.synchronize()
    dev = dict(o=_np(o), S_T=_np(S_T), dq=_np(q.grad), dk=_np(k.grad), dv=_np(v.grad), dg=_np(g.grad),
               dbeta=_np(beta.grad), dS0=_np(S0.grad))
    ref = Hn.run_oracle(case)
    res = Hn.compare(dev, ref, names=tuple(dev))
    print(res, flush=True)
    Hn.assert_parity(res, Hn.TOL["f32"], case.name)


def test_autograd_output_only_delta_bf16():
    # DeltaNet member (no g), zero initial state, loss on o alone
    from paper_2608_12700_amd.autograd import gated_delta_rule
    case = W.make_case("bf16_autograd_delta", B=1, T=200, H=2, dk=128, dv=64, variant="delta",
                       S0_std=0.0, dST_std=0.0)
    print("case", W.describe(case), flush=True)
    t = Hn.device_inputs(case)
    q, k, v, beta = (_leaf(t[n]) for n in ("q", "k", "v", "beta"))
    o, _ = gated_delta_rule(q, k, v, None, beta, None, variant="delta")
    (o.float() * t["dO"].float()).sum().backward()
    torch.cuda.synchronize()
    dev = dict(o=_np(o), dq=_np(q.grad), dk=_np(k.grad), dv=_np(v.grad), dbeta=_np(beta.grad))
    ref = Hn.run_oracle(case)
    res = Hn.compare(dev, ref, names=tuple(dev))
    print(res, flush=True)
    Hn.assert_parity(res, Hn.TOL["bf16"], case.name)


def test_graph_capture_replay_bitwise():
    from paper_2608_12700_amd import gdn
    case = W.make_case("bf16_graph", B=2, T=200, H=3, dk=128, dv=128)
    print("case", W.describe(case), flush=True)
    t = Hn.device_inputs(case)
    dev = t["q"].device
    p = gdn.make_problem(case.B, case.T, case.H, case.dk, case.dv)
    nch = gdn.gdn_num_chunks(p)
    outs = dict(o=torch.empty_like(t["v"]),
                S_T=torch.empty((case.B, case.H, case.dk, case.dv), dtype=torch.float32, device=dev),
                states=torch.empty((nch, case.H, case.dk, case.dv), dtype=torch.float32, device=dev),
                dq=torch.empty_like(t["q"]), dk=torch.empty_like(t["k"]), dv=torch.empty_like(t["v"]),
                dg=torch.empty_like(t["g"]), dbeta=torch.empty_like(t["beta"]), dS0=torch.empty_like(t["S0"]))
    wsf = torch.empty(gdn.gdn_fwd_workspace_size(p), dtype=torch.uint8, device=dev)
    wsb = torch.empty(gdn.gdn_bwd_workspace_size(p), dtype=torch.uint8, device=dev)
    P = lambda x: ctypes.c_void_p(x.data_ptr())

    def step():
        s = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        assert gdn.gdn_fwd(p, P(t["q"]), P(t["k"]), P(t["v"]), P(t["g"]), P(t["beta"]), P(t["S0"]),
                           P(outs["o"]), P(outs["S_T"]), P(outs["states"]), P(wsf), wsf.numel(), s) == 0
        assert gdn.gdn_bwd(p, P(t["q"]), P(t["k"]), P(t["v"]), P(t["g"]), P(t["beta"]), P(outs["states"]),
                           P(t["dO"]), P(t["dS_T"]), P(outs["dq"]), P(outs["dk"]), P(outs["dv"]),
                           P(outs["dg"]), P(outs["dbeta"]), P(outs["dS0"]), P(wsb), wsb.numel(), s) == 0

    step()
    torch.cuda.synchronize()
    eager = {n: x.clone() for n, x in outs.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm the side stream before capture
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
        # eager work between replays
        step()
        torch.cuda.synchronize()
        for n, x in outs.items():
            assert torch.equal(x.view(torch.uint8), eager[n].view(torch.uint8)), ("eager", rep, n)
    print("4 replays bitwise equal to eager", flush=True)


class _GDNLayer(torch.nn.Module):
    """x -> projections -> gated delta rule (HIP) -> output projection."""

    def __init__(self, D, H, dk, dv, variant="gated_delta"):
        super().__init__()
        self.H, self.dk, self.dv, self.variant = H, dk, dv, variant
        self.wq = torch.nn.Linear(D, H * dk, bias=False)
        self.wk = torch.nn.Linear(D, H * dk, bias=False)
        self.wv = torch.nn.Linear(D, H * dv, bias=False)
        self.wg = torch.nn.Linear(D, H)
        self.wb = torch.nn.Linear(D, H)
        self.wo = torch.nn.Linear(H * dv, D, bias=False)

    def forward(self, x):
        from paper_2608_12700_amd.autograd import gated_delta_rule
        B, L, _ = x.shape
        q = F.normalize(self.wq(x).view(B, L, self.H, self.dk), dim=-1)
        k = F.normalize(self.wk(x).view(B, L, self.H, self.dk), dim=-1)
        v = self.wv(x).view(B, L, self.H, self.dv)
        g = -0.1 * F.softplus(self.wg(x))
        beta = torch.sigmoid(self.wb(x))
        if self.variant == "decay_only":
            # the scalar-decay (SSD) member: no erase, so keep the state's growth
            # in check with the key scale
            beta = None
            k = k * 0.5
        bf = torch.bfloat16
        c = lambda t: None if t is None else t.float().contiguous()
        o, _ = gated_delta_rule(q.to(bf).contiguous(), k.to(bf).contiguous(), v.to(bf).contiguous(),
                                c(g), c(beta), variant=self.variant)
        return self.wo(o.float().reshape(B, L, self.H * self.dv))


@pytest.mark.parametrize("variant", ["gated_delta", "decay_only"])
def test_training_smoke_l256(variant):
    """300 Adam steps at L = 256: the gated delta rule and the scalar-decay (SSD)
    member, both through the native forward and backward."""
    torch.manual_seed(0)
    dev = torch.device("cuda")
    D, H, dk, dv, B, L = 64, 2, 64, 64, 4, 256
    teacher = _GDNLayer(D, H, dk, dv, variant).to(dev)
    student = _GDNLayer(D, H, dk, dv, variant).to(dev)
    for prm in teacher.parameters():
        prm.requires_grad_(False)
    opt = torch.optim.Adam(student.parameters(), lr=3e-3)
    losses = []  # MSE relative to the teacher output's mean square
    for it in range(300):
        x = torch.randn(B, L, D, device=dev)
        with torch.no_grad():
            y = teacher(x)
            scale = y.pow(2).mean()
        loss = F.mse_loss(student(x), y) / scale
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
        losses.append(loss.item())
        assert np.isfinite(losses[-1]), (it, losses[-1])
    first, last = np.mean(losses[:10]), np.mean(losses[-10:])
    print(f"training smoke {variant}: relative loss {first:.4f} -> {last:.4f}", flush=True)
    assert last < 0.2 * first, (first, last)

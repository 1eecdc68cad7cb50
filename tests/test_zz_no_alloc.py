"""gdn_fwd_noalloc (the forward with its workspace in the library's fixed
device array) against gdn_fwd with a caller workspace, through the C ABI: two
calls in a row, the second on a smaller problem, must both reproduce gdn_fwd's
outputs bit for bit (the same kernels run on the same inputs).  A problem whose
workspace exceeds the array is rejected before anything runs."""
import ctypes

import numpy as np
import pytest

import workloads as W
from tests import harness as Hn

pytestmark = pytest.mark.gpu


def _outputs(case, dev):
    import torch
    p_nch = W.total_chunks_for(case.B, case.T, cu_seqlens=case.cu_seqlens)
    act = torch.bfloat16 if case.io_dtype == "bf16" else torch.float32
    return dict(o=torch.full((case.B, case.T, case.H, case.dv), float("nan"), dtype=act, device=dev),
                S_T=torch.full((case.N, case.H, case.dk, case.dv), float("nan"), device=dev),
                states=torch.full((p_nch, case.H, case.dk, case.dv), float("nan"), device=dev))


def _fwd_both(case):
    import torch
    from paper_2608_12700_amd import gdn
    dev = torch.device("cuda")
    t = Hn.device_inputs(case)
    packed = None if case.cu_seqlens is None else gdn.Packed(case.cu_seqlens, dev)
    io = gdn.GDN_BF16 if case.io_dtype == "bf16" else gdn.GDN_F32
    p = (gdn.make_problem(case.B, case.T, case.H, case.dk, case.dv, io_dtype=io, variant=case.variant)
         if packed is None else
         gdn.make_problem(case.B, case.T, case.H, case.dk, case.dv, io_dtype=io, variant=case.variant,
                          cu_host=packed.host, cu_dev_ptr=packed.dev.data_ptr()))
    assert gdn.gdn_fwd_workspace_size(p) <= gdn.NOALLOC_SCRATCH_BYTES
    X = lambda x: None if x is None else ctypes.c_void_p(x.data_ptr())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    ref, got = _outputs(case, dev), _outputs(case, dev)
    ws = torch.empty(gdn.gdn_fwd_workspace_size(p), dtype=torch.uint8, device=dev)
    rc = gdn.gdn_fwd(p, X(t["q"]), X(t["k"]), X(t["v"]), X(t["g"]), X(t["beta"]), X(t["S0"]), X(ref["o"]),
                     X(ref["S_T"]), X(ref["states"]), X(ws), ws.numel(), s)
    assert rc == 0, gdn.STATUS.get(rc)
    rc = gdn.gdn_fwd_noalloc(p, X(t["q"]), X(t["k"]), X(t["v"]), X(t["g"]), X(t["beta"]), X(t["S0"]),
                             X(got["o"]), X(got["S_T"]), X(got["states"]), s)
    assert rc == 0, gdn.STATUS.get(rc)
    torch.cuda.synchronize()
    return ref, got


def _check(case):
    import torch
    print("case", W.describe(case), flush=True)
    ref, got = _fwd_both(case)
    for nm in ref:
        assert torch.equal(ref[nm].view(torch.uint8), got[nm].view(torch.uint8)), (case.name, nm)
    # and the shared output against the float64 oracle, to the usual bar
    oracle = Hn.run_oracle(case)
    dev = {nm: x.float().cpu().numpy().astype(np.float64) for nm, x in got.items()}
    res = Hn.compare(dev, oracle, names=("o", "S_T", "states"))
    Hn.assert_parity(res, Hn.TOL[case.io_dtype], case.name)


def test_two_calls_second_smaller():
    # a larger problem, then a smaller one that reuses the array's stale contents
    _check(W.make_case("noalloc_big", B=2, T=1000, H=4, dk=128, dv=128, seed=3))
    _check(W.make_case("noalloc_small", B=1, T=130, H=2, dk=64, dv=64, io_dtype="f32", seed=4))


def test_packed_and_members():
    cu = np.array([0, 5, 70, 200], np.int32)
    _check(W.make_case("noalloc_packed", B=1, T=200, H=3, dk=64, dv=256, cu_seqlens=cu, seed=5))
    _check(W.make_case("noalloc_delta", B=1, T=150, H=2, dk=128, dv=64, variant="delta", seed=6))


def test_too_large_rejected_untouched():
    import torch
    from paper_2608_12700_amd import gdn
    p = gdn.make_problem(4, 4096, 16, 128, 128)  # ~360 MB of workspace
    assert gdn.gdn_fwd_workspace_size(p) > gdn.NOALLOC_SCRATCH_BYTES
    o = torch.zeros(8, device="cuda")
    X = lambda x: ctypes.c_void_p(x.data_ptr())
    rc = gdn.gdn_fwd_noalloc(p, X(o), X(o), X(o), X(o), X(o), None, X(o), X(o), X(o),
                             ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == -10
    torch.cuda.synchronize()
    assert bool((o == 0).all())

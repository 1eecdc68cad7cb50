"""The Python binding rejects bad dtypes and shapes before any library call
(CPU only).  The tensors here live on the CPU: every call must raise from the
binding's own checks (dtype, then shape, then device), so nothing reaches the
C ABI and no pointer to host memory is ever handed to a kernel."""
import pytest
import torch

from paper_2608_12700_amd import gdn

B, T, H, DK, DV = 2, 70, 3, 64, 64
NCH = B * 2


def _fwd_args(dt=torch.bfloat16):
    return dict(q=torch.zeros(B, T, H, DK, dtype=dt), k=torch.zeros(B, T, H, DK, dtype=dt),
                v=torch.zeros(B, T, H, DV, dtype=dt), g=torch.zeros(B, T, H), beta=torch.zeros(B, T, H),
                S0=torch.zeros(B, H, DK, DV))


def _bwd_args(dt=torch.bfloat16):
    a = _fwd_args(dt)
    del a["S0"]
    a["chunk_states"] = torch.zeros(NCH, H, DK, DV)
    a["dO"] = torch.zeros(B, T, H, DV, dtype=dt)
    a["dS_T"] = torch.zeros(B, H, DK, DV)
    return a


def _call_fwd(a):
    return gdn.fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S0"])


def _call_bwd(a):
    return gdn.bwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["chunk_states"], a["dO"], a["dS_T"])


@pytest.mark.parametrize("dt", [torch.float16, torch.float64, torch.int32])
def test_unsupported_activation_dtypes_rejected(dt):
    with pytest.raises(TypeError, match="bfloat16 or torch.float32"):
        _call_fwd(_fwd_args(dt))
    with pytest.raises(TypeError, match="bfloat16 or torch.float32"):
        _call_bwd(_bwd_args(dt))


def test_mixed_dtypes_rejected():
    a = _fwd_args()
    a["k"] = a["k"].float()
    with pytest.raises(TypeError, match="k must be"):
        _call_fwd(a)
    a = _fwd_args()
    a["g"] = a["g"].double()
    with pytest.raises(TypeError, match="g must be"):
        _call_fwd(a)


@pytest.mark.parametrize("name,shape", [
    ("k", (B, T, H, DK - 1)), ("v", (B, T - 1, H, DV)), ("g", (B, T, H + 1)), ("beta", (B, T)),
    ("S0", (B, H, DK, DV // 2)), ("S0", (B + 1, H, DK, DV)),
])
def test_fwd_shapes_checked(name, shape):
    a = _fwd_args()
    a[name] = torch.zeros(shape, dtype=a[name].dtype)
    with pytest.raises(ValueError, match="shape"):
        _call_fwd(a)


@pytest.mark.parametrize("name,shape", [
    ("dO", (B, T, H, DV + 8)), ("chunk_states", (NCH - 1, H, DK, DV)),
    ("chunk_states", (NCH, H, DK, DV + 1)), ("dS_T", (B, H, DK, 1)), ("beta", (B, T, H - 1)),
])
def test_bwd_shapes_checked(name, shape):
    a = _bwd_args()
    a[name] = torch.zeros(shape, dtype=a[name].dtype)
    with pytest.raises(ValueError, match="shape"):
        _call_bwd(a)


def test_q_must_be_4d():
    a = _fwd_args()
    a["q"] = torch.zeros(B * T, H, DK, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match=r"\[B, T, H, d_k\]"):
        _call_fwd(a)


def test_packed_chunk_states_sized_from_offsets():
    cu = [0, 5, 70, 70, 140]  # 1 + 2 + 0 + 2 chunks
    q = torch.zeros(1, 140, H, DK, dtype=torch.bfloat16)
    v = torch.zeros(1, 140, H, DV, dtype=torch.bfloat16)
    g = torch.zeros(1, 140, H)
    st = torch.zeros(4, H, DK, DV)  # one short
    with pytest.raises(ValueError, match="chunk_states must have shape"):
        gdn.bwd(q, q, v, g, g, st, v, None, cu_seqlens=cu)


def test_channelwise_gate_shapes_checked():
    a = _fwd_args(torch.float32)
    g = torch.zeros(B, T, H, DK)
    w = torch.zeros(B, T, H, DV + 1)
    with pytest.raises(ValueError, match="w must have shape"):
        gdn.cw_fwd(a["q"], a["k"], a["v"], g, None, w)
    with pytest.raises(ValueError, match="g must have shape"):
        gdn.cw_fwd(a["q"], a["k"], a["v"], torch.zeros(B, T, H), None, None)


def test_host_tensors_never_reach_the_library():
    # well-formed but on the CPU: refused before any C call
    with pytest.raises(ValueError, match="GPU device"):
        _call_fwd(_fwd_args())
    with pytest.raises(ValueError, match="GPU device"):
        _call_bwd(_bwd_args())

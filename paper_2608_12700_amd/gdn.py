"""Python binding of libgdn.so (argument marshalling only).

Every step of the forward and backward runs in the library's HIP kernels; this
module allocates outputs and workspace with torch, fills the C structs and
passes raw device pointers plus the current HIP stream.  If the library has not
been built, every entry point raises: there is no fallback.

Names mirror the C ABI in include/gdn.h:
  gdn_fwd(...) / gdn_bwd(...)       raw calls on pointers (ctypes)
  fwd(...) / bwd(...)               torch-tensor conveniences built on them
  gdn_cw_fwd / gdn_cw_bwd,          the channel-wise members (per-channel g, b, w)
  cw_fwd(...) / cw_bwd(...)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgdn.so")

GDN_OK = 0
STATUS = {0: "GDN_OK", -1: "GDN_ERR_NULL", -2: "GDN_ERR_SHAPE", -3: "GDN_ERR_UNSUPPORTED",
          -4: "GDN_ERR_DTYPE", -5: "GDN_ERR_WORKSPACE", -6: "GDN_ERR_ALIAS", -7: "GDN_ERR_VARLEN",
          -8: "GDN_ERR_HIP", -9: "GDN_ERR_VARIANT", -10: "GDN_ERR_TOO_LARGE"}
NOALLOC_SCRATCH_BYTES = 64 << 20  # GDN_NOALLOC_SCRATCH_BYTES
GDN_F32, GDN_BF16 = 0, 1
VARIANTS = {"gated_delta": 0, "delta": 1, "decay_only": 2}
CHUNK = 64


class GdnError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {STATUS.get(code, code)}")
        self.code = code


class Problem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
        ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
        ("num_seqs", ctypes.c_int32),
        ("cu_seqlens_host", ctypes.POINTER(ctypes.c_int32)),
        ("cu_seqlens_dev", ctypes.c_void_p),
        ("io_dtype", ctypes.c_int), ("variant", ctypes.c_int),
    ]


EXPORTED = ("gdn_num_chunks", "gdn_fwd_workspace_size", "gdn_bwd_workspace_size", "gdn_fwd",
            "gdn_bwd", "gdn_fwd_ex", "gdn_bwd_ex", "gdn_cw_fwd_workspace_size",
            "gdn_cw_bwd_workspace_size", "gdn_cw_fwd", "gdn_cw_bwd", "gdn_cw_fwd_ex", "gdn_cw_bwd_ex",
            "gdn_status_str", "gdn_version", "gdn_fwd_noalloc")
CW_BWD_STAGES = ("cw_bwd_prep", "cw_bwd_scan", "cw_bwd_grad_v", "cw_bwd_grad_d")
NUM_STAGES = 4
FWD_STAGES = ("fwd_prep", "fwd_scan", "fwd_exact", None)  # the output is fused into the scan
BWD_STAGES = ("bwd_prep", "bwd_scan", "bwd_grad", "bwd_exact")

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libgdn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_12700_amd.build`")
    lib = ctypes.CDLL(path)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    P = ctypes.POINTER(Problem)
    lib.gdn_num_chunks.argtypes = [P]
    lib.gdn_num_chunks.restype = ctypes.c_int64
    lib.gdn_fwd_workspace_size.argtypes = [P]
    lib.gdn_fwd_workspace_size.restype = sz
    lib.gdn_bwd_workspace_size.argtypes = [P]
    lib.gdn_bwd_workspace_size.restype = sz
    lib.gdn_fwd.argtypes = [P] + [vp] * 9 + [vp, sz, vp]
    lib.gdn_fwd.restype = ctypes.c_int
    lib.gdn_bwd.argtypes = [P] + [vp] * 14 + [vp, sz, vp]
    lib.gdn_bwd.restype = ctypes.c_int
    lib.gdn_fwd_ex.argtypes = [P] + [vp] * 9 + [vp, sz, vp, vp]
    lib.gdn_fwd_ex.restype = ctypes.c_int
    lib.gdn_bwd_ex.argtypes = [P] + [vp] * 14 + [vp, sz, vp, vp]
    lib.gdn_bwd_ex.restype = ctypes.c_int
    lib.gdn_cw_fwd_workspace_size.argtypes = [P]
    lib.gdn_cw_fwd_workspace_size.restype = sz
    lib.gdn_cw_bwd_workspace_size.argtypes = [P]
    lib.gdn_cw_bwd_workspace_size.restype = sz
    lib.gdn_cw_fwd.argtypes = [P] + [vp] * 10 + [vp, sz, vp]
    lib.gdn_cw_fwd.restype = ctypes.c_int
    lib.gdn_cw_bwd.argtypes = [P] + [vp] * 16 + [vp, sz, vp]
    lib.gdn_cw_bwd.restype = ctypes.c_int
    lib.gdn_cw_fwd_ex.argtypes = [P] + [vp] * 10 + [vp, sz, vp, vp]
    lib.gdn_cw_fwd_ex.restype = ctypes.c_int
    lib.gdn_cw_bwd_ex.argtypes = [P] + [vp] * 16 + [vp, sz, vp, vp]
    lib.gdn_cw_bwd_ex.restype = ctypes.c_int
    lib.gdn_fwd_noalloc.argtypes = [P] + [vp] * 9 + [vp]
    lib.gdn_fwd_noalloc.restype = ctypes.c_int
    lib.gdn_status_str.argtypes = [ctypes.c_int]
    lib.gdn_status_str.restype = ctypes.c_char_p
    lib.gdn_version.argtypes = []
    lib.gdn_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def make_problem(B, T, H, dk, dv, *, io_dtype=GDN_BF16, variant="gated_delta", cu_host=None,
                 cu_dev_ptr=None, chunk=CHUNK):
    """Fill a gdn_problem.  ``cu_host`` is an int32 numpy array kept alive by the caller."""
    p = Problem()
    p.B, p.T, p.H, p.dk, p.dv, p.chunk = B, T, H, dk, dv, chunk
    if cu_host is not None:
        p.num_seqs = len(cu_host) - 1
        p.cu_seqlens_host = cu_host.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        p.cu_seqlens_dev = cu_dev_ptr
    else:
        p.num_seqs = B
        p.cu_seqlens_host = None
        p.cu_seqlens_dev = None
    p.io_dtype = io_dtype
    p.variant = VARIANTS[variant] if isinstance(variant, str) else int(variant)
    return p


# --- raw C-ABI calls (same names as the C functions) -----------------------

def gdn_num_chunks(p: Problem) -> int:
    return int(load().gdn_num_chunks(ctypes.byref(p)))


def gdn_fwd_workspace_size(p: Problem) -> int:
    return int(load().gdn_fwd_workspace_size(ctypes.byref(p)))


def gdn_bwd_workspace_size(p: Problem) -> int:
    return int(load().gdn_bwd_workspace_size(ctypes.byref(p)))


def gdn_fwd(p, q, k, v, g, beta, S0, o, S_T, states, ws, ws_bytes, stream) -> int:
    return int(load().gdn_fwd(ctypes.byref(p), q, k, v, g, beta, S0, o, S_T, states, ws, ws_bytes,
                              stream))


def gdn_bwd(p, q, k, v, g, beta, states, dO, dS_T, dq, dk, dv, dg, dbeta, dS0, ws, ws_bytes,
            stream) -> int:
    return int(load().gdn_bwd(ctypes.byref(p), q, k, v, g, beta, states, dO, dS_T, dq, dk, dv, dg,
                              dbeta, dS0, ws, ws_bytes, stream))


def gdn_fwd_noalloc(p, q, k, v, g, beta, S0, o, S_T, states, stream) -> int:
    return int(load().gdn_fwd_noalloc(ctypes.byref(p), q, k, v, g, beta, S0, o, S_T, states, stream))


def gdn_fwd_ex(p, q, k, v, g, beta, S0, o, S_T, states, ws, ws_bytes, stream, events) -> int:
    return int(load().gdn_fwd_ex(ctypes.byref(p), q, k, v, g, beta, S0, o, S_T, states, ws, ws_bytes,
                                 stream, events))


def gdn_bwd_ex(p, q, k, v, g, beta, states, dO, dS_T, dq, dk, dv, dg, dbeta, dS0, ws, ws_bytes,
               stream, events) -> int:
    return int(load().gdn_bwd_ex(ctypes.byref(p), q, k, v, g, beta, states, dO, dS_T, dq, dk, dv, dg,
                                 dbeta, dS0, ws, ws_bytes, stream, events))


def gdn_cw_fwd_workspace_size(p: Problem) -> int:
    return int(load().gdn_cw_fwd_workspace_size(ctypes.byref(p)))


def gdn_cw_bwd_workspace_size(p: Problem) -> int:
    return int(load().gdn_cw_bwd_workspace_size(ctypes.byref(p)))


def gdn_cw_fwd(p, q, k, v, g, b, w, S0, o, S_T, states, ws, ws_bytes, stream) -> int:
    return int(load().gdn_cw_fwd(ctypes.byref(p), q, k, v, g, b, w, S0, o, S_T, states, ws, ws_bytes, stream))


def gdn_cw_bwd(p, q, k, v, g, b, w, states, dO, dS_T, dq, dk, dv, dg, db, dw, dS0, ws, ws_bytes,
               stream) -> int:
    return int(load().gdn_cw_bwd(ctypes.byref(p), q, k, v, g, b, w, states, dO, dS_T, dq, dk, dv, dg, db, dw,
                                 dS0, ws, ws_bytes, stream))


def gdn_cw_fwd_ex(p, q, k, v, g, b, w, S0, o, S_T, states, ws, ws_bytes, stream, events) -> int:
    return int(load().gdn_cw_fwd_ex(ctypes.byref(p), q, k, v, g, b, w, S0, o, S_T, states, ws, ws_bytes,
                                    stream, events))


def gdn_cw_bwd_ex(p, q, k, v, g, b, w, states, dO, dS_T, dq, dk, dv, dg, db, dw, dS0, ws, ws_bytes,
                  stream, events) -> int:
    return int(load().gdn_cw_bwd_ex(ctypes.byref(p), q, k, v, g, b, w, states, dO, dS_T, dq, dk, dv, dg, db,
                                    dw, dS0, ws, ws_bytes, stream, events))


def gdn_status_str(code: int) -> str:
    return load().gdn_status_str(code).decode()


def gdn_version() -> str:
    return load().gdn_version().decode()


# --- torch conveniences ----------------------------------------------------

def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _check(t: torch.Tensor, name: str, dtype, device, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _io_dtype(q: torch.Tensor):
    """The activation dtype code of q: bf16 or fp32 only."""
    if not isinstance(q, torch.Tensor):
        raise TypeError(f"q must be a torch.Tensor, got {type(q).__name__}")
    if q.dtype == torch.bfloat16:
        return GDN_BF16
    if q.dtype == torch.float32:
        return GDN_F32
    raise TypeError(f"activations must be torch.bfloat16 or torch.float32, got {q.dtype}")


def _dims(q, v):
    """(B, T, H, dk, dv) from q [B,T,H,dk] and v [B,T,H,dv]."""
    if q.dim() != 4:
        raise ValueError(f"q must be [B, T, H, d_k], got shape {tuple(q.shape)}")
    if not isinstance(v, torch.Tensor) or v.dim() != 4:
        raise ValueError(f"v must be [B, T, H, d_v], got shape {tuple(getattr(v, 'shape', ()))}")
    B, T, H, dk = q.shape
    return B, T, H, dk, v.shape[-1]


def _num_chunks(B, T, packed):
    if packed is None:
        return B * (-(-T // CHUNK))
    cu = [int(x) for x in packed.host]
    return sum(-(-max(cu[n + 1] - cu[n], 0) // CHUNK) for n in range(len(cu) - 1))


def _on_gpu(q):
    if q.device.type != "cuda":
        raise ValueError(f"tensors must be on a GPU device, got {q.device}: the library reads device memory")


class Packed:
    """Packed sequence offsets: a host int32 copy and a device int32 copy."""

    def __init__(self, cu_seqlens, device):
        import numpy as np
        if isinstance(cu_seqlens, torch.Tensor):
            host = cu_seqlens.detach().to("cpu", torch.int32).numpy()
        else:
            host = np.asarray(cu_seqlens, dtype=np.int32)
        self.host = np.ascontiguousarray(host, dtype=np.int32)
        self.dev = torch.from_numpy(self.host).to(device)

    @property
    def num_seqs(self) -> int:
        return len(self.host) - 1


def _problem_for(q, v, variant, packed: Optional[Packed]):
    B, T, H, dk, dv = _dims(q, v)
    io = _io_dtype(q)
    if packed is None:
        return make_problem(B, T, H, dk, dv, io_dtype=io, variant=variant)
    return make_problem(B, T, H, dk, dv, io_dtype=io, variant=variant, cu_host=packed.host,
                        cu_dev_ptr=packed.dev.data_ptr())


def fwd(q, k, v, g, beta, S0=None, *, variant="gated_delta", cu_seqlens=None, workspace=None):
    """Forward: returns (o, S_T, chunk_states).  See include/gdn.h for layouts."""
    dev = q.device
    packed = None if cu_seqlens is None else (cu_seqlens if isinstance(cu_seqlens, Packed)
                                              else Packed(cu_seqlens, dev))
    p = _problem_for(q, v, variant, packed)
    B, T, H, dk, dv = _dims(q, v)
    N = p.num_seqs
    for name, t, shp in (("q", q, (B, T, H, dk)), ("k", k, (B, T, H, dk)), ("v", v, (B, T, H, dv))):
        _check(t, name, q.dtype, dev, shp)
    for name, t, shp in (("g", g, (B, T, H)), ("beta", beta, (B, T, H)), ("S0", S0, (N, H, dk, dv))):
        if t is not None:
            _check(t, name, torch.float32, dev, shp)
    _on_gpu(q)
    nch = gdn_num_chunks(p)
    if nch < 0:
        raise GdnError(nch, "gdn_num_chunks")
    o = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    S_T = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    states = torch.empty((nch, H, dk, dv), dtype=torch.float32, device=dev)
    wsb = gdn_fwd_workspace_size(p)
    ws = workspace if workspace is not None else torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    rc = gdn_fwd(p, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(o), _ptr(S_T),
                 _ptr(states), _ptr(ws), ws.numel(), ctypes.c_void_p(_stream_handle(dev)))
    if rc != GDN_OK:
        raise GdnError(rc, "gdn_fwd")
    return o, S_T, states


def bwd(q, k, v, g, beta, chunk_states, dO, dS_T=None, *, variant="gated_delta", cu_seqlens=None,
        workspace=None):
    """Backward: returns (dq, dk, dv, dg, dbeta, dS0); dg / dbeta are None when the variant has no g / beta."""
    dev = q.device
    packed = None if cu_seqlens is None else (cu_seqlens if isinstance(cu_seqlens, Packed)
                                              else Packed(cu_seqlens, dev))
    p = _problem_for(q, v, variant, packed)
    B, T, H, dk, dv = _dims(q, v)
    N = p.num_seqs
    nch = _num_chunks(B, T, packed)
    for name, t, shp in (("q", q, (B, T, H, dk)), ("k", k, (B, T, H, dk)), ("v", v, (B, T, H, dv)),
                         ("dO", dO, (B, T, H, dv))):
        _check(t, name, q.dtype, dev, shp)
    _check(chunk_states, "chunk_states", torch.float32, dev, (nch, H, dk, dv))
    for name, t, shp in (("g", g, (B, T, H)), ("beta", beta, (B, T, H)), ("dS_T", dS_T, (N, H, dk, dv))):
        if t is not None:
            _check(t, name, torch.float32, dev, shp)
    _on_gpu(q)
    dq = torch.empty_like(q)
    dk_ = torch.empty_like(k)
    dvv = torch.empty_like(v)
    dg = None if g is None else torch.empty((B, T, H), dtype=torch.float32, device=dev)
    db = None if beta is None else torch.empty((B, T, H), dtype=torch.float32, device=dev)
    dS0 = torch.empty((N, H, dk, dv), dtype=torch.float32, device=dev)
    wsb = gdn_bwd_workspace_size(p)
    ws = workspace if workspace is not None else torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    rc = gdn_bwd(p, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(chunk_states), _ptr(dO),
                 _ptr(dS_T), _ptr(dq), _ptr(dk_), _ptr(dvv), _ptr(dg), _ptr(db), _ptr(dS0), _ptr(ws),
                 ws.numel(), ctypes.c_void_p(_stream_handle(dev)))
    if rc != GDN_OK:
        raise GdnError(rc, "gdn_bwd")
    return dq, dk_, dvv, dg, db, dS0


def _packed_of(cu_seqlens, dev):
    if cu_seqlens is None:
        return None
    return cu_seqlens if isinstance(cu_seqlens, Packed) else Packed(cu_seqlens, dev)


def cw_fwd(q, k, v, g=None, b=None, w=None, S0=None, *, cu_seqlens=None, workspace=None):
    """Channel-wise forward: returns (o, S_T, chunk_states).  q, k, v fp32 or bf16 (o follows);
    g, b [B,T,H,d_k] and w [B,T,H,d_v] fp32, each may be None (neutral gate).  See include/gdn.h."""
    dev = q.device
    packed = _packed_of(cu_seqlens, dev)
    p = _problem_for(q, v, "gated_delta", packed)
    B, T, H, dk, dv = _dims(q, v)
    N = p.num_seqs
    for name, t, shp in (("q", q, (B, T, H, dk)), ("k", k, (B, T, H, dk)), ("v", v, (B, T, H, dv))):
        _check(t, name, q.dtype, dev, shp)
    for name, t, shp in (("g", g, (B, T, H, dk)), ("b", b, (B, T, H, dk)), ("w", w, (B, T, H, dv)),
                         ("S0", S0, (N, H, dk, dv))):
        if t is not None:
            _check(t, name, torch.float32, dev, shp)
    _on_gpu(q)
    nch = gdn_num_chunks(p)
    if nch < 0:
        raise GdnError(nch, "gdn_num_chunks")
    o = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    S_T = torch.empty((p.num_seqs, H, dk, dv), dtype=torch.float32, device=dev)
    states = torch.empty((nch, H, dk, dv), dtype=torch.float32, device=dev)
    wsb = gdn_cw_fwd_workspace_size(p)
    ws = workspace if workspace is not None else torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    rc = gdn_cw_fwd(p, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(b), _ptr(w), _ptr(S0), _ptr(o), _ptr(S_T),
                    _ptr(states), _ptr(ws), ws.numel(), ctypes.c_void_p(_stream_handle(dev)))
    if rc != GDN_OK:
        raise GdnError(rc, "gdn_cw_fwd")
    return o, S_T, states


def cw_bwd(q, k, v, g, b, w, chunk_states, dO, dS_T=None, *, cu_seqlens=None, workspace=None):
    """Channel-wise backward: returns (dq, dk, dv, dg, db, dw, dS0); dq, dk, dv in the dtype of q,
    a gate's gradient (fp32) is None when the gate is None."""
    dev = q.device
    packed = _packed_of(cu_seqlens, dev)
    p = _problem_for(q, v, "gated_delta", packed)
    B, T, H, dk, dv = _dims(q, v)
    N = p.num_seqs
    nch = _num_chunks(B, T, packed)
    for name, t, shp in (("q", q, (B, T, H, dk)), ("k", k, (B, T, H, dk)), ("v", v, (B, T, H, dv)),
                         ("dO", dO, (B, T, H, dv))):
        _check(t, name, q.dtype, dev, shp)
    _check(chunk_states, "chunk_states", torch.float32, dev, (nch, H, dk, dv))
    for name, t, shp in (("g", g, (B, T, H, dk)), ("b", b, (B, T, H, dk)), ("w", w, (B, T, H, dv)),
                         ("dS_T", dS_T, (N, H, dk, dv))):
        if t is not None:
            _check(t, name, torch.float32, dev, shp)
    _on_gpu(q)
    like = lambda t: None if t is None else torch.empty_like(t)
    dq, dk_, dvv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    dg, db, dw = like(g), like(b), like(w)
    dS0 = torch.empty((p.num_seqs, H, dk, dv), dtype=torch.float32, device=dev)
    wsb = gdn_cw_bwd_workspace_size(p)
    ws = workspace if workspace is not None else torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    rc = gdn_cw_bwd(p, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(b), _ptr(w), _ptr(chunk_states), _ptr(dO),
                    _ptr(dS_T), _ptr(dq), _ptr(dk_), _ptr(dvv), _ptr(dg), _ptr(db), _ptr(dw), _ptr(dS0),
                    _ptr(ws), ws.numel(), ctypes.c_void_p(_stream_handle(dev)))
    if rc != GDN_OK:
        raise GdnError(rc, "gdn_cw_bwd")
    return dq, dk_, dvv, dg, db, dw, dS0


__all__ = ["load", "make_problem", "Problem", "Packed", "GdnError", "fwd", "bwd", "gdn_fwd", "gdn_bwd",
           "gdn_fwd_ex", "gdn_bwd_ex", "gdn_fwd_noalloc", "NOALLOC_SCRATCH_BYTES", "NUM_STAGES", "FWD_STAGES", "BWD_STAGES",
           "gdn_num_chunks", "gdn_fwd_workspace_size", "gdn_bwd_workspace_size", "gdn_status_str",
           "gdn_version", "EXPORTED", "LIB_PATH", "VARIANTS", "cw_fwd", "cw_bwd", "gdn_cw_fwd", "gdn_cw_bwd",
           "gdn_cw_fwd_ex", "gdn_cw_bwd_ex", "gdn_cw_fwd_workspace_size", "gdn_cw_bwd_workspace_size",
           "CW_BWD_STAGES"]

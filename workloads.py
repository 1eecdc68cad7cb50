"""Seeded synthetic workloads for the gated-delta-rule forward/backward.

This module draws inputs only. It holds none of the recurrence's arithmetic, so
that both the float64 oracle and the HIP path can consume the same bits without
sharing any code that computes the method.

Draw recipe (fixed order, one ``numpy.random.Generator(PCG64(seed))`` per case):
  q, k, v, beta_logit, g_raw, S0, dO, dS_T, then the non-finite injection sites.
Every tensor is drawn in float64, q and k are L2-normalised per (token, head)
in float64, beta = sigmoid(beta_logit), g = -c * softplus(g_raw).  Each tensor
is then rounded once to float32 (round to nearest even) and, for bf16 I/O, the
activations q, k, v, dO once more to bfloat16 (round to nearest even).  Gates,
states and their gradients stay float32.  The arrays returned are float32 and
hold exactly the rounded values, so the oracle (which upcasts them to float64)
and the device (which receives the same bits) see identical inputs.

Layouts (token-major, row-major): q, k [B, T, H, dk]; v, dO [B, T, H, dv];
g, beta [B, T, H]; S0, dS_T [N, H, dk, dv] with N = B, or N = number of packed
sequences when ``cu_seqlens`` is given (then B = 1).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

VARIANTS = ("gated_delta", "delta", "decay_only")


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round a float32 array to the nearest bfloat16 value (ties to even).

    Returns float32 holding bf16-representable values. NaN stays NaN and
    +-Inf stays +-Inf.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    r = ((u + bias) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).copy()
    nan = np.isnan(x)
    out[nan] = np.float32("nan")
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-representable."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def _softplus(z: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, z)


def _sigmoid(z: np.ndarray) -> np.ndarray:
    return 0.5 * (1.0 + np.tanh(0.5 * z))


def varlen_lengths(rng: np.random.Generator, n: int, total: int, lo: int, hi: int) -> np.ndarray:
    """Lengths uniform in [lo, hi], rescaled to sum exactly to ``total``.

    1. draw L_i ~ U{lo..hi};
    2. L_i <- clamp(round(L_i * total / sum L), lo, hi);
    3. hand out the residual +-1 cyclically in index order to entries that stay
       inside [lo, hi] until the sum is ``total``.
    """
    if not (n * lo <= total <= n * hi):
        raise ValueError("total length out of reach of the bounds")
    L = rng.integers(lo, hi + 1, size=n).astype(np.int64)
    L = np.clip(np.rint(L * (total / L.sum())).astype(np.int64), lo, hi)
    i = 0
    while L.sum() != total:
        step = 1 if L.sum() < total else -1
        if lo <= L[i] + step <= hi:
            L[i] += step
        i = (i + 1) % n
    return L


@dataclasses.dataclass
class Case:
    """One concrete synthetic problem (all arrays float32, see module doc)."""

    name: str
    variant: str
    io_dtype: str  # "f32" or "bf16"
    B: int
    T: int
    H: int
    dk: int
    dv: int
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: Optional[np.ndarray]
    beta: Optional[np.ndarray]
    S0: np.ndarray
    dO: np.ndarray
    dS_T: np.ndarray
    cu_seqlens: Optional[np.ndarray] = None
    chunk: int = 64
    injected: Optional[dict] = None

    @property
    def N(self) -> int:
        return self.B if self.cu_seqlens is None else len(self.cu_seqlens) - 1

    def seq_bounds(self):
        """List of (batch row, token start, length) per sequence."""
        if self.cu_seqlens is None:
            return [(b, 0, self.T) for b in range(self.B)]
        cu = self.cu_seqlens
        return [(0, int(cu[n]), int(cu[n + 1] - cu[n])) for n in range(len(cu) - 1)]

    def total_chunks(self) -> int:
        return sum(-(-L // self.chunk) for (_, _, L) in self.seq_bounds())


def make_case(
    name: str,
    *,
    B: int,
    T: int,
    H: int,
    dk: int,
    dv: int,
    io_dtype: str = "bf16",
    variant: str = "gated_delta",
    decay_scale: float = 0.1,
    S0_std: float = 0.1,
    dST_std: float = 1.0,
    seed: int = 0,
    cu_seqlens: Optional[np.ndarray] = None,
    inject: Optional[str] = None,
    normalize_qk: bool = True,
) -> Case:
    """Draw one case. ``S0_std`` / ``dST_std`` of 0 give exact zeros.

    ``inject``: None, "row" (NaN over a whole v[b,t,h,:] row and +Inf in one g
    entry) or "elem" (NaN in one element of v and +Inf in one g entry).
    """
    if variant not in VARIANTS:
        raise ValueError(variant)
    if io_dtype not in ("f32", "bf16"):
        raise ValueError(io_dtype)
    rng = np.random.Generator(np.random.PCG64(seed))
    N = B if cu_seqlens is None else len(cu_seqlens) - 1

    def draw(shape):
        return rng.standard_normal(shape)  # float64

    def normed(x):
        nrm = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
        return x / nrm

    def to_f32(x):
        return np.asarray(x, dtype=np.float32)

    def act(x):
        x = to_f32(x)
        return round_bf16(x) if io_dtype == "bf16" else x

    q = draw((B, T, H, dk))
    if normalize_qk:
        q = normed(q)
    q = act(q)
    k = draw((B, T, H, dk))
    if normalize_qk:
        k = normed(k)
    k = act(k)
    v = act(draw((B, T, H, dv)))
    beta = to_f32(_sigmoid(draw((B, T, H))))
    g = to_f32(-decay_scale * _softplus(draw((B, T, H))))
    # S0 and dS_T are always drawn so that the draw order does not depend on
    # whether they are used; a zero standard deviation then gives exact +0.
    S0 = draw((N, H, dk, dv))
    S0 = to_f32(S0_std * S0) if S0_std > 0 else np.zeros((N, H, dk, dv), np.float32)
    dO = act(draw((B, T, H, dv)))
    dST = draw((N, H, dk, dv))
    dST = to_f32(dST_std * dST) if dST_std > 0 else np.zeros((N, H, dk, dv), np.float32)

    injected = None
    if inject is not None:
        b1, t1, h1 = int(rng.integers(B)), int(rng.integers(T)), int(rng.integers(H))
        j1 = int(rng.integers(dv))
        b2, t2, h2 = int(rng.integers(B)), int(rng.integers(T)), int(rng.integers(H))
        if inject == "row":
            v[b1, t1, h1, :] = np.float32("nan")
        elif inject == "elem":
            v[b1, t1, h1, j1] = np.float32("nan")
        else:
            raise ValueError(inject)
        g[b2, t2, h2] = np.float32("inf")
        injected = {"v_nan": (b1, t1, h1, j1 if inject == "elem" else None), "g_inf": (b2, t2, h2)}

    if variant == "delta":
        g = None
    if variant == "decay_only":
        beta = None
    return Case(
        name=name, variant=variant, io_dtype=io_dtype, B=B, T=T, H=H, dk=dk, dv=dv,
        q=q, k=k, v=v, g=g, beta=beta, S0=S0, dO=dO, dS_T=dST,
        cu_seqlens=None if cu_seqlens is None else np.asarray(cu_seqlens, np.int32),
        injected=injected,
    )


# The five workloads the path is specified on (shapes, distributions, seeds).
def config0() -> Case:
    """fp32, B=1, T=256, H=2, dk=dv=64, S0=0, dS_T=0 (small parity case)."""
    return make_case("fp32_B1_T256_H2_d64", B=1, T=256, H=2, dk=64, dv=64, io_dtype="f32",
                     S0_std=0.0, dST_std=0.0)


def config1() -> Case:
    """bf16 I/O, fp32 state: B=4, T=4096, H=16, dk=dv=128 (the throughput workload)."""
    return make_case("bf16_B4_T4096_H16_d128", B=4, T=4096, H=16, dk=128, dv=128)


def config2(T: int = 65536) -> Case:
    """Long-sequence reverse-state stress: B=1, H=16, d=128, g=-0.02*softplus."""
    return make_case(f"bf16_B1_T{T}_H16_d128_long", B=1, T=T, H=16, dk=128, dv=128,
                     decay_scale=0.02)


def config3(kind: str) -> Case:
    """Family variants at B=8, T=2048, H=32, d=64: 'delta', 'decay_only', 'nan_row', 'nan_elem'."""
    common = dict(B=8, T=2048, H=32, dk=64, dv=64)
    if kind == "delta":
        return make_case("bf16_B8_T2048_H32_d64_delta", variant="delta", **common)
    if kind == "decay_only":
        return make_case("bf16_B8_T2048_H32_d64_decay", variant="decay_only", decay_scale=1.0, **common)
    if kind in ("nan_row", "nan_elem"):
        return make_case(f"bf16_B8_T2048_H32_d64_{kind}", inject=kind.split("_")[1], **common)
    raise ValueError(kind)


def config4_cu_seqlens(seed: int = 0) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    L = varlen_lengths(rng, 16, 32768, 64, 4096)
    return np.concatenate([[0], np.cumsum(L)]).astype(np.int32)


def config4() -> Case:
    """Packed varlen: 16 sequences, T=32768 total, H=16, dk=128, dv=256."""
    cu = config4_cu_seqlens()
    return make_case("bf16_varlen16_T32768_H16_dk128_dv256", B=1, T=int(cu[-1]), H=16, dk=128,
                     dv=256, cu_seqlens=cu)


def total_chunks_for(B: int, T: int, chunk: int = 64, cu_seqlens=None) -> int:
    if cu_seqlens is None:
        return B * (-(-T // chunk))
    cu = np.asarray(cu_seqlens)
    return int(sum(-(-int(cu[n + 1] - cu[n]) // chunk) for n in range(len(cu) - 1)))


def describe(case: Case) -> str:
    return (f"{case.name}: variant={case.variant} io={case.io_dtype} B={case.B} T={case.T} "
            f"H={case.H} dk={case.dk} dv={case.dv} N={case.N}")


# ---------------------------------------------------------------------------
# Channel-wise members: per-channel gates g, b [B,T,H,dk] and w [B,T,H,dv].
# Draw order (one PCG64(seed) per case): q, k, v, g_raw, b_logit, w_logit, S0,
# dO, dS_T.  g = -decay * softplus(g_raw) (a log-decay per channel, mean about
# -0.8 * decay), b = sigmoid(b_logit), w = 1.5 * sigmoid(w_logit); q, k are
# L2-normalised per (token, head).  Everything is rounded once to float32.
# ``gates`` names the gates present: "gbw" (full GDN), "kda" (b = w = a scalar
# beta per token broadcast over the channels, g per channel), "g" (GLA), ""
# (LA).  Absent gates are None.  For bf16 I/O the activations q, k, v, dO are
# rounded once more to bfloat16 (RNE); gates and states stay fp32.
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class CwCase:
    name: str
    B: int
    T: int
    H: int
    dk: int
    dv: int
    gates: str
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: Optional[np.ndarray]
    b: Optional[np.ndarray]
    w: Optional[np.ndarray]
    S0: np.ndarray
    dO: np.ndarray
    dS_T: np.ndarray
    cu_seqlens: Optional[np.ndarray] = None
    io_dtype: str = "f32"

    @property
    def N(self) -> int:
        return self.B if self.cu_seqlens is None else len(self.cu_seqlens) - 1


def make_cw_case(name, B, T, H, dk, dv, *, gates="gbw", seed=0, decay=1.0, cu_seqlens=None,
                 S0_std=0.1, dST_std=1.0, io_dtype="f32") -> CwCase:
    if cu_seqlens is not None:
        assert B == 1 and int(cu_seqlens[-1]) == T
    rng = np.random.Generator(np.random.PCG64(seed))
    N = B if cu_seqlens is None else len(cu_seqlens) - 1
    f32 = lambda x: np.ascontiguousarray(x, dtype=np.float32)

    def normed(x):
        return x / np.linalg.norm(x, axis=-1, keepdims=True)

    q = f32(normed(rng.standard_normal((B, T, H, dk))))
    k = f32(normed(rng.standard_normal((B, T, H, dk))))
    v = f32(rng.standard_normal((B, T, H, dv)))
    g_raw = rng.standard_normal((B, T, H, dk))
    b_logit = rng.standard_normal((B, T, H, dk))
    w_logit = rng.standard_normal((B, T, H, dv))
    S0 = f32(S0_std * rng.standard_normal((N, H, dk, dv)))
    dO = f32(rng.standard_normal((B, T, H, dv)))
    dS_T = f32(dST_std * rng.standard_normal((N, H, dk, dv)))
    # decay: a scale of the log-decay, one number or one per token (shape [T])
    dscale = np.asarray(decay, dtype=np.float64)
    if dscale.ndim == 1:
        dscale = dscale[None, :, None, None]
    g = f32(-dscale * _softplus(g_raw)) if gates in ("gbw", "kda", "g") else None
    b = w = None
    if gates == "gbw":
        b = f32(_sigmoid(b_logit))
        w = f32(1.5 * _sigmoid(w_logit))
    elif gates == "kda":
        beta = f32(_sigmoid(b_logit[..., 0]))
        b = f32(np.repeat(beta[..., None], dk, axis=-1))
        w = f32(np.repeat(beta[..., None], dv, axis=-1))
    if io_dtype == "bf16":
        q, k, v, dO = (round_bf16(x) for x in (q, k, v, dO))
    elif io_dtype != "f32":
        raise ValueError(f"io_dtype {io_dtype!r}")
    return CwCase(name, B, T, H, dk, dv, gates, q, k, v, g, b, w, S0, dO, dS_T,
                  None if cu_seqlens is None else np.asarray(cu_seqlens, dtype=np.int32), io_dtype)


__all__ = [
    "CwCase", "make_cw_case",
    "VARIANTS", "Case", "make_case", "round_bf16", "bf16_bits", "varlen_lengths",
    "config0", "config1", "config2", "config3", "config4", "config4_cu_seqlens",
    "total_chunks_for", "describe",
]

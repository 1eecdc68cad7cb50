"""torch.autograd wrapper of the gated-delta-rule forward and backward.

``gated_delta_rule(q, k, v, g, beta, S0)`` returns ``(o, S_T)`` and records a
node whose backward is one ``gdn_bwd`` call: the only tensor saved between the
two is the forward's ``chunk_states`` (the state before every chunk of 64
tokens), as the C ABI prescribes.  Argument marshalling only -- both
directions run entirely in the library's HIP kernels (``gdn.fwd`` /
``gdn.bwd``), and a missing library raises.

The loss the backward differentiates is whatever the caller builds from
``o`` and ``S_T``; autograd hands the backward ``dO = dL/do`` and
``dS_T = dL/dS_T`` (zeros for an output that does not reach the loss).
Gradients are returned for q, k, v, g, beta and S0 (None where the input is
None: ``g`` for the DeltaNet member, ``beta`` for the scalar-decay member,
``S0`` when the sequence starts from the zero state).

``channelwise_rule`` does the same for the channel-wise members (per-channel
g, b, w; ``gdn.cw_fwd`` / ``gdn.cw_bwd``).
"""
from __future__ import annotations

from typing import Optional

import torch

from . import gdn


class GatedDeltaRule(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, g, beta, S0, variant, cu_seqlens):
        o, S_T, states = gdn.fwd(q, k, v, g, beta, S0, variant=variant, cu_seqlens=cu_seqlens)
        ctx.save_for_backward(q, k, v, g, beta, states)
        ctx.variant = variant
        ctx.cu_seqlens = cu_seqlens
        ctx.has_S0 = S0 is not None
        return o, S_T

    @staticmethod
    def backward(ctx, dO, dS_T):
        q, k, v, g, beta, states = ctx.saved_tensors
        dO = dO.contiguous()
        dS_T = None if dS_T is None else dS_T.contiguous()
        dq, dk, dv, dg, db, dS0 = gdn.bwd(q, k, v, g, beta, states, dO, dS_T, variant=ctx.variant,
                                          cu_seqlens=ctx.cu_seqlens)
        return dq, dk, dv, dg, db, (dS0 if ctx.has_S0 else None), None, None


def gated_delta_rule(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: Optional[torch.Tensor] = None,
                     beta: Optional[torch.Tensor] = None, S0: Optional[torch.Tensor] = None, *,
                     variant: str = "gated_delta", cu_seqlens=None):
    """(o, S_T) of the recurrence S_t = (I - beta_t k_t k_t^T) e^{g_t} S_{t-1} + beta_t k_t v_t^T,
    o_t = S_t^T q_t, differentiable in every tensor argument.  Layouts and dtypes as
    ``gdn.fwd``: q, k [B,T,H,d_k] and v [B,T,H,d_v] in bf16 or fp32 (contiguous), g and
    beta [B,T,H] fp32, S0 [N,H,d_k,d_v] fp32."""
    return GatedDeltaRule.apply(q, k, v, g, beta, S0, variant, cu_seqlens)


class ChannelwiseRule(torch.autograd.Function):
    """The channel-wise members (per-channel g, b, w; bf16 or fp32 activations, fp32
    gates): one gdn_cw_fwd and one gdn_cw_bwd."""

    @staticmethod
    def forward(ctx, q, k, v, g, b, w, S0, cu_seqlens):
        o, S_T, states = gdn.cw_fwd(q, k, v, g, b, w, S0, cu_seqlens=cu_seqlens)
        ctx.save_for_backward(q, k, v, g, b, w, states)
        ctx.cu_seqlens = cu_seqlens
        ctx.has_S0 = S0 is not None
        return o, S_T

    @staticmethod
    def backward(ctx, dO, dS_T):
        q, k, v, g, b, w, states = ctx.saved_tensors
        dO = dO.contiguous()
        dS_T = None if dS_T is None else dS_T.contiguous()
        dq, dk, dv, dg, db, dw, dS0 = gdn.cw_bwd(q, k, v, g, b, w, states, dO, dS_T, cu_seqlens=ctx.cu_seqlens)
        return dq, dk, dv, dg, db, dw, (dS0 if ctx.has_S0 else None), None


def channelwise_rule(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: Optional[torch.Tensor] = None,
                     b: Optional[torch.Tensor] = None, w: Optional[torch.Tensor] = None,
                     S0: Optional[torch.Tensor] = None, *, cu_seqlens=None):
    """(o, S_T) of S_t = (I - k_t (b_t * k_t)^T) Diag(e^{g_t}) S_{t-1} + k_t (w_t * v_t)^T,
    o_t = S_t^T q_t, differentiable in every tensor argument.  Contiguous: q, k
    [B,T,H,d_k] and v [B,T,H,d_v] in bf16 or fp32 (one dtype; o and the activation
    gradients follow it); g, b [B,T,H,d_k], w [B,T,H,d_v] and S0 [N,H,d_k,d_v] fp32.
    A gate left None is
    neutral (g = 0, b = 0, w = 1): KDA passes b = w = beta broadcast over the
    channels, GLA passes g alone, LA none."""
    return ChannelwiseRule.apply(q, k, v, g, b, w, S0, cu_seqlens)


__all__ = ["GatedDeltaRule", "gated_delta_rule", "ChannelwiseRule", "channelwise_rule"]

"""The masked pipeline boundary as an in-graph autograd op (paper Sec. 3.1;
Alg. 1).

Forward, at a masked boundary: the sender keeps K of the H values of every
token with the shared mask g(layer, step, B, S, H) and transmits only those;
the receiver scatters them back (scaled) into a dense activation.  Backward
inherits the same sparsity: the receiver packs the incoming gradient at the
same positions (same key, so the same mask), the sender scatters it back, so
dL/dh = scale * (dL/dh~ ⊙ m) and masked positions get exactly zero.

BoundarySend / BoundaryRecv are the two halves, for a sender and a receiver
on different pipeline stages (the packed values are what crosses the link in
both directions); masked_boundary chains them on one device.  The scale is
applied wherever a payload is unpacked, in both directions (the receiver of
each direction absorbs it): the backward payload is the unscaled packed
gradient, and the pair together gives exactly dL/dh = scale * (dL/dh~ ⊙ m).
Use the two halves as a pair.  Every
operation is a library call (ac_mask_pack, ac_unpack_scatter); this module
only wires them into autograd.
"""
from __future__ import annotations

import torch

from . import ac_keep_count, ac_mask_pack, ac_unpack_scatter, make_key


def boundary_key(seed: int, layer: int, step: int, microbatch: int, h: torch.Tensor):
    """The mask key of a [B, S, H] activation at boundary `layer`, step `step`."""
    B, S, H = h.shape
    return make_key(seed=seed, layer=layer, step=step, microbatch=microbatch, B=B, S=S, H=H)


class BoundarySend(torch.autograd.Function):
    """Sender side: h [B, S, H] -> packed values [B*S, K] (what is sent).
    Backward: the packed gradient received from the next stage is scattered
    into a dense gradient of h (scaled, zeros off the mask)."""

    @staticmethod
    def forward(ctx, h: torch.Tensor, K: int, key, scale: float):
        B, S, H = h.shape
        vals, idx = ac_mask_pack(h.reshape(B * S, H), K, key)
        ctx.key, ctx.scale, ctx.shape = key, float(scale), (B, S, H)
        ctx.save_for_backward(idx)
        ctx.mark_non_differentiable(idx)
        return vals, idx

    @staticmethod
    def backward(ctx, g_vals: torch.Tensor, _g_idx):
        (idx,) = ctx.saved_tensors
        B, S, H = ctx.shape
        g = ac_unpack_scatter(g_vals.contiguous(), H, ctx.key, ctx.scale, idx=idx)
        return g.view(B, S, H), None, None, None


class BoundaryRecv(torch.autograd.Function):
    """Receiver side: packed values [B*S, K] -> dense scale * (h ⊙ m)
    [B, S, H].  Backward: the gradient of the dense activation is packed at
    the same positions (what is sent back)."""

    @staticmethod
    def forward(ctx, vals: torch.Tensor, idx, shape, key, scale: float):
        B, S, H = shape
        y = ac_unpack_scatter(vals.contiguous(), H, key, float(scale), idx=idx)
        ctx.key, ctx.K, ctx.shape = key, vals.shape[1], (B, S, H)
        return y.view(B, S, H)

    @staticmethod
    def backward(ctx, g_y: torch.Tensor):
        B, S, H = ctx.shape
        g_vals, _ = ac_mask_pack(g_y.contiguous().reshape(B * S, H), ctx.K, ctx.key, with_idx=False)
        return g_vals, None, None, None, None


def masked_boundary(h: torch.Tensor, keep: float, key, scale=None) -> torch.Tensor:
    """scale * (h ⊙ m) with K = round(keep * H) kept per token; gradients
    flow through the same mask.  scale defaults to H / K (unbiased for a
    fixed-K mask; the paper's 1 / (1 - p) differs from it by < 0.5% at the
    configurations used here)."""
    H = h.shape[-1]
    K = ac_keep_count(H, keep)
    s = H / K if scale is None else float(scale)
    vals, idx = BoundarySend.apply(h, K, key, s)
    return BoundaryRecv.apply(vals, idx, tuple(h.shape), key, s)

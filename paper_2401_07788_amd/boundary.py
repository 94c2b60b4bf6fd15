"""A pipeline-stage boundary inside one process (Sec. 2.1, Fig. 1): the
activation crossing it is compressed by the library's sender and
reconstructed by its receiver in the forward pass, and its gradient the same
way in the backward pass, so that a model can be trained with the
compression the boundary would apply between two devices.

TopK (Sec. 2.3) compresses both directions, optionally with an error
feedback buffer per direction (Sec. 2.4).  The gradient is sent either at
the indices the activation's TopK kept (Sec. 3.2, the mode the GPT-2 runs
needed) or through a TopK of its own.  Every step runs in the HIP library;
this module only moves tensors and keeps the buffers."""
from __future__ import annotations

import torch

from . import tc


class _TopkBoundaryFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, k_fwd, k_bwd, e_fwd, e_bwd, reuse):
        n_seg = x.shape[0]
        x2 = x.detach().reshape(n_seg, -1).contiguous()
        L = x2.shape[1]
        if e_fwd is not None:
            pl = tc.ef_step_topk(x2, e_fwd, k_fwd, n_seg)
        else:
            pl = tc.topk_compress(x2, k_fwd, n_seg)
        y = tc.topk_decompress(pl, L)
        ctx.pl = pl
        ctx.meta = (n_seg, L, k_bwd, e_bwd, reuse, x.shape)
        return y.view(x.shape)

    @staticmethod
    def backward(ctx, gy):
        n_seg, L, k_bwd, e_bwd, reuse, shape = ctx.meta
        g2 = gy.reshape(n_seg, L).contiguous()
        if reuse:
            val = tc.topk_gather(ctx.pl, g2, e=e_bwd)
            gx = tc.topk_decompress(ctx.pl._replace(val=val), L)
        elif e_bwd is not None:
            gx = tc.topk_decompress(tc.ef_step_topk(g2, e_bwd, k_bwd, n_seg), L)
        else:
            gx = tc.topk_decompress(tc.topk_compress(g2, k_bwd, n_seg), L)
        ctx.pl = None
        return gx.view(shape), None, None, None, None, None


class TopkBoundary(torch.nn.Module):
    """TopK K% per segment (dim 0 of the tensor: samples or token rows) in both
    directions.  num/den: the kept fraction (k = ceil(seg_len * num / den));
    ef: an error feedback buffer per direction, created at the first call and
    carried across calls (reset() clears them); reuse_indices: the gradient
    goes at the activation's kept indices instead of a TopK of its own."""

    def __init__(self, num: int, den: int, ef: bool = False, reuse_indices: bool = True):
        super().__init__()
        self.num, self.den, self.ef, self.reuse = num, den, ef, reuse_indices
        self.e_fwd = self.e_bwd = None

    def reset(self):
        self.e_fwd = self.e_bwd = None

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        n_seg = x.shape[0]
        L = x.numel() // n_seg
        k = tc.topk_count(L, self.num, self.den)
        if self.ef and (self.e_fwd is None or self.e_fwd.numel() != x.numel() or self.e_fwd.device != x.device):
            self.e_fwd = torch.zeros(x.numel(), dtype=torch.float32, device=x.device)
            self.e_bwd = torch.zeros(x.numel(), dtype=torch.float32, device=x.device)
        return _TopkBoundaryFn.apply(x, k, k, self.e_fwd if self.ef else None, self.e_bwd if self.ef else None,
                                     self.reuse)

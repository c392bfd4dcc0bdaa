"""Drop-in autograd activation (Listing 1): the forward saves only the packed
b-bit interval indices; the backward multiplies by the stored values."""
from __future__ import annotations

import torch

from ._lib import ACTS, Table, Weight, W_NORMAL, bwd, fit_table, fwd


class FewBitActivation(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, table: Table):
        x = x.contiguous()
        y, codes = fwd(table, x)
        ctx.save_for_backward(codes)
        ctx.table = table
        return y

    @staticmethod
    def backward(ctx, grad_out):
        (codes,) = ctx.saved_tensors
        grad_in = bwd(ctx.table, grad_out.contiguous(), codes)
        return grad_in, None


class FewBitAct(torch.nn.Module):
    """Few-bit GELU / SiLU / Sigmoid / Tanh / ReLU / SELU / Softplus.

    The table is fitted once at construction (Sec. 3); by default under a
    standard normal weight on [-10, 10] with a 4000-cell grid, optionally
    refined by gradient descent on the boundaries.
    """

    def __init__(self, act: str = "gelu", bits: int = 3, weight: Weight | None = None,
                 n_grid: int = 4000, table: Table | None = None, refine: bool = False):
        super().__init__()
        self.act = act
        self.bits = bits
        if table is None:
            weight = weight or Weight(W_NORMAL, -10.0, 10.0)
            table = fit_table(ACTS[act], bits, weight, n_grid, refine=refine)
        self.table = table

    def forward(self, x):
        return FewBitActivation.apply(x, self.table)

    def extra_repr(self) -> str:
        return f"act={self.act}, bits={self.bits}"

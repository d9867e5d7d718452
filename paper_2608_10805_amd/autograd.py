"""torch.autograd wrapper and nn.Module around the fused WTConv library.

Only x and the parameters are saved for backward (no per-level subband
tensors): the backward kernel recomputes both Haar pyramids on chip.
"""
import math

import torch

from . import binding


class WTConvFunction(torch.autograd.Function):
    """y = WTConv(x; base_w, base_scale, base_bias, level_w[0..L-1], level_scale[0..L-1]),
    base_bias optional (None)."""

    @staticmethod
    def forward(ctx, x, base_w, base_scale, base_bias, *level_params):
        L = len(level_params) // 2
        level_w, level_scale = list(level_params[:L]), list(level_params[L:])
        x = x.contiguous()
        y = binding.forward(x, base_w, base_scale, level_w, level_scale, bias=base_bias)
        ctx.save_for_backward(x, base_w, base_scale, base_bias, *level_params)
        ctx.L = L
        return y

    @staticmethod
    def backward(ctx, dy):
        x, base_w, base_scale, base_bias, *level_params = ctx.saved_tensors
        L = ctx.L
        need_dbias = base_bias is not None and ctx.needs_input_grad[3]
        out = binding.backward(x, dy.contiguous(), base_w, base_scale, level_params[:L], level_params[L:],
                               need_dx=ctx.needs_input_grad[0], bias=base_bias, need_dbias=need_dbias)
        dx, dbw, dbs, dlw, dls = out[:5]
        dbb = out[5] if need_dbias else None
        return (dx, dbw, dbs, dbb, *dlw, *dls)


def wtconv(x, base_w, base_scale, level_w, level_scale, base_bias=None):
    return WTConvFunction.apply(x, base_w, base_scale, base_bias, *level_w, *level_scale)


class WTConv2d(torch.nn.Module):
    """Drop-in depthwise replacement: k x k base conv plus an L-level Haar branch.

    Parameters are float32 whatever the activation dtype. Initialisation follows
    the synthetic recipe of the tests (uniform kernels, base scale 1, small
    level scales) and can be overwritten freely.
    """

    def __init__(self, channels: int, kernel_size: int = 5, levels: int = 1, bias: bool = False, device=None):
        super().__init__()
        C, k = channels, kernel_size
        bound = 1.0 / math.sqrt(k * k)
        self.base_w = torch.nn.Parameter(torch.empty(C, k, k, device=device).uniform_(-bound, bound))
        self.base_scale = torch.nn.Parameter(torch.ones(C, device=device))
        self.base_bias = torch.nn.Parameter(torch.zeros(C, device=device)) if bias else None
        self.level_w = torch.nn.ParameterList(
            [torch.nn.Parameter(torch.empty(4 * C, k, k, device=device).uniform_(-bound, bound))
             for _ in range(levels)])
        self.level_scale = torch.nn.ParameterList(
            [torch.nn.Parameter(torch.full((4 * C,), 0.1, device=device)) for _ in range(levels)])

    def forward(self, x):
        return wtconv(x, self.base_w, self.base_scale, list(self.level_w), list(self.level_scale), self.base_bias)

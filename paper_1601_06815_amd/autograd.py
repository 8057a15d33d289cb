"""torch.autograd binding of the OaA convolution layer.

Training needs the forward convolution and the two backward convolutions
(arXiv:1601.06815, Section 3.2); ``OaAConv2dFunction`` connects them to
autograd and ``OaAConv2d`` holds a weight like a layer. Argument marshalling
only: every pass runs in the library's kernels through ``binding.Plan``.

The layer computes a true convolution (the kernel flipped), valid output,
stride 1: y = OaAConv2d(x) equals torch's cross-correlation
``conv2d(x, w.flip(-1, -2))``.

Spectra cached by a plan belong to the last pass it ran. The backward pass
reuses the kernel and input spectra of its own forward pass when the plan has
run nothing since (its ``generation`` counter, which every pass of the plan
advances, is unchanged), and recomputes them from the saved tensors
otherwise.
"""

import math

import torch

from . import binding


class OaAConv2dFunction(torch.autograd.Function):
    """y = conv(x, w) through ``plan`` (a binding.Plan of matching shape)."""

    @staticmethod
    def forward(ctx, x, w, plan):
        x, w = x.contiguous(), w.contiguous()
        y = plan.forward(x, w)
        ctx.generation = plan.generation
        ctx.plan = plan
        ctx.save_for_backward(x, w)
        return y

    @staticmethod
    def backward(ctx, gy):
        x, w = ctx.saved_tensors
        plan = ctx.plan
        gy = gy.contiguous()
        need_x, need_w = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
        if not (need_x or need_w):
            return None, None, None
        fresh = plan.generation == ctx.generation
        # both gradients start from the gradient windows transformed here
        # (which the fused passes do not keep: they transform them again)
        dx = plan.backward_data(gy, None if fresh else w)
        dw = (plan.backward_filter(None if fresh else x, None if plan.caches_grad_spectra else gy)
              if need_w else None)
        return (dx if need_x else None), dw, None


class OaAConv2d(torch.nn.Module):
    """Convolution layer with K = out_channels kernels of side kernel_size over
    C = in_channels channels; one plan (and device workspace) per input shape.
    ``tiling`` is passed to binding.Plan ("auto", "paper" or (L, b))."""

    def __init__(self, in_channels, out_channels, kernel_size, tiling="auto", device="cuda"):
        super().__init__()
        self.C, self.K, self.n = in_channels, out_channels, kernel_size
        self.tiling = tiling
        std = math.sqrt(1.0 / (in_channels * kernel_size * kernel_size))
        self.weight = torch.nn.Parameter(
            torch.randn(out_channels, in_channels, kernel_size, kernel_size, device=device) * std)
        self._plans = {}

    def plan_for(self, B, N):
        key = (B, N, self.weight.device)
        if key not in self._plans:
            self._plans[key] = binding.Plan(B, self.C, self.K, N, self.n, device=self.weight.device,
                                            tiling=self.tiling)
        return self._plans[key]

    def forward(self, x):
        B, C, N, N2 = x.shape
        if C != self.C or N != N2:
            raise ValueError(f"expected x[B,{self.C},N,N], got {tuple(x.shape)}")
        return OaAConv2dFunction.apply(x, self.weight, self.plan_for(B, N))

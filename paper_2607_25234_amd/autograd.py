"""torch.autograd wrappers of the WHTMix C ABI (argument marshalling only).

    y = whtmix_mix(x, gain)                                  # joint gain G[N_pad, C]
    y = whtmix_mix_separable(x, log_gain_tokens, log_gain_channels)

The forward and backward passes both run in the HIP kernels of libwhtmix.so
(whtmix_forward*/whtmix_backward*); gradients flow to x and to the gains, as
when the paper trains the mixer (section IV-A).
"""
from __future__ import annotations

import torch

from . import whtmix


class WHTMixFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, gain):
        x = x.contiguous()
        gain = gain.contiguous()
        ctx.save_for_backward(x, gain)
        return whtmix.forward(x, gain)

    @staticmethod
    def backward(ctx, dy):
        x, gain = ctx.saved_tensors
        dx, dgain = whtmix.backward(x, dy.contiguous(), gain,
                                    want_dx=ctx.needs_input_grad[0],
                                    want_dgain=ctx.needs_input_grad[1])
        return dx, dgain


class WHTMixSeparableFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, log_gain_tokens, log_gain_channels):
        x = x.contiguous()
        gt = log_gain_tokens.contiguous()
        gc = log_gain_channels.contiguous()
        ctx.save_for_backward(x, gt, gc)
        return whtmix.forward_separable(x, gt, gc)

    @staticmethod
    def backward(ctx, dy):
        x, gt, gc = ctx.saved_tensors
        want_g = ctx.needs_input_grad[1] or ctx.needs_input_grad[2]
        dx, dgt, dgc = whtmix.backward_separable(x, dy.contiguous(), gt, gc,
                                                 want_dx=ctx.needs_input_grad[0],
                                                 want_dgains=want_g)
        return dx, dgt, dgc


def whtmix_mix(x, gain):
    """Differentiable y = H_N (G o (H_N x H_C)) H_C."""
    return WHTMixFunction.apply(x, gain)


def whtmix_mix_separable(x, log_gain_tokens, log_gain_channels):
    """Differentiable eq. (2) then eq. (3) with log-domain gains."""
    return WHTMixSeparableFunction.apply(x, log_gain_tokens, log_gain_channels)

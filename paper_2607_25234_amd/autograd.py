"""torch.autograd wrappers of the WHTMix C ABI (argument marshalling only).

    y = whtmix_mix(x, gain)                                  # joint gain G[N_pad, C]
    y = whtmix_mix_separable(x, log_gain_tokens, log_gain_channels)
    y = whtmix_block(x, w_in, gain, w_out)                   # eqs. (1)-(4)
    y = whtmix_block_separable(x, w_in, log_gain_tokens, log_gain_channels, w_out)

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


class WHTMixBlockFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w_in, gain, w_out):
        x, w_in, gain, w_out = (t.contiguous() for t in (x, w_in, gain, w_out))
        ctx.save_for_backward(x, w_in, gain, w_out)
        return whtmix.module_forward(x, w_in, gain, w_out)

    @staticmethod
    def backward(ctx, dy):
        x, w_in, gain, w_out = ctx.saved_tensors
        dx, dwi, dwo, dg = whtmix.module_backward(x, w_in, gain, w_out, dy.contiguous(),
                                                  want_dgain=ctx.needs_input_grad[2])
        return dx, dwi.to(w_in.dtype), dg, dwo.to(w_out.dtype)


class WHTMixBlockSeparableFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w_in, log_gain_tokens, log_gain_channels, w_out):
        x, w_in, gt, gc, w_out = (t.contiguous() for t in
                                  (x, w_in, log_gain_tokens, log_gain_channels, w_out))
        ctx.save_for_backward(x, w_in, gt, gc, w_out)
        return whtmix.module_forward_separable(x, w_in, gt, gc, w_out)

    @staticmethod
    def backward(ctx, dy):
        x, w_in, gt, gc, w_out = ctx.saved_tensors
        want_g = ctx.needs_input_grad[2] or ctx.needs_input_grad[3]
        dx, dwi, dwo, dgt, dgc = whtmix.module_backward_separable(
            x, w_in, gt, gc, w_out, dy.contiguous(), want_dgains=want_g)
        return dx, dwi.to(w_in.dtype), dgt, dgc, dwo.to(w_out.dtype)


def whtmix_block(x, w_in, gain, w_out):
    """Differentiable block of eqs. (1)-(4): mixer(x W_in) W_out (joint gain).
    Weight gradients are computed in float32 and returned in the weights' dtype."""
    return WHTMixBlockFunction.apply(x, w_in, gain, w_out)


def whtmix_block_separable(x, w_in, log_gain_tokens, log_gain_channels, w_out):
    """Differentiable block with the paper's log-domain gains."""
    return WHTMixBlockSeparableFunction.apply(x, w_in, log_gain_tokens, log_gain_channels, w_out)


def whtmix_mix(x, gain):
    """Differentiable y = H_N (G o (H_N x H_C)) H_C."""
    return WHTMixFunction.apply(x, gain)


def whtmix_mix_separable(x, log_gain_tokens, log_gain_channels):
    """Differentiable eq. (2) then eq. (3) with log-domain gains."""
    return WHTMixSeparableFunction.apply(x, log_gain_tokens, log_gain_channels)

"""Autograd node of the soft codeword (Sec. 3.5) and its BCJR-STE variant.

``BcjrQuant`` wraps the library's entry points as a ``torch.autograd.Function``:

* soft mode: forward ``bcjr_soft_codeword`` (the soft codeword at temperature
  T), backward ``bcjr_soft_codeword_vjp``;
* hard mode (BCJR-STE, Sec. "BCJR-STE variant"): forward ``viterbi_decode``
  (the hard minimum-distortion codeword), backward ``bcjr_ste_vjp``, i.e. the
  exact gradient of the temperature-T relaxation in place of an identity
  straight-through gradient.

T is a plain number read at call time (a detached schedule value, Sec. 3.5),
so it gets no gradient.  Gradients flow to the weights and, if it requires
grad, to the codebook.  Every step runs in the library's HIP kernels.
"""
from __future__ import annotations

import torch

from . import bcjr_soft_codeword, bcjr_soft_codeword_vjp, bcjr_ste_vjp, viterbi_decode

__all__ = ["BcjrQuant", "bcjr_quant"]


def _temperature(T) -> float:
    if isinstance(T, torch.Tensor):
        if T.numel() != 1:
            raise ValueError("T must be a scalar")
        T = T.detach().item()
    return float(T)


class BcjrQuant(torch.autograd.Function):
    """w[B, L] -> codeword[B, L] (soft at T, or hard Viterbi when ``hard``)."""

    @staticmethod
    def forward(ctx, w, codebook, state_bits, k, T, hard):
        T = _temperature(T)
        w = w.contiguous()
        codebook = codebook.contiguous()
        if hard:
            _, out = viterbi_decode(w, codebook, state_bits, k)
        else:
            out, _ = bcjr_soft_codeword(w, codebook, state_bits, k, T, want_logZ=False)
        ctx.state_bits, ctx.k, ctx.T, ctx.hard = state_bits, k, T, bool(hard)
        ctx.save_for_backward(w, codebook, out if hard else None)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        w, codebook, w_hard = ctx.saved_tensors
        need_w, need_c = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
        if not (need_w or need_c):
            return None, None, None, None, None, None
        g = grad_out.contiguous()
        n, k, T = ctx.state_bits, ctx.k, ctx.T
        if ctx.hard:
            dW, dc = bcjr_ste_vjp(w, codebook, n, k, T, w_hard, g, want_dW=need_w,
                                  want_dCodebook=need_c)
        else:
            dW, dc = bcjr_soft_codeword_vjp(w, codebook, n, k, T, g, want_dW=need_w,
                                            want_dCodebook=need_c)
        return dW, dc, None, None, None, None


def bcjr_quant(W, codebook, state_bits: int, k: int, T, block: int = 256, hard: bool = False):
    """Quantise a float32 tensor of any shape as consecutive blocks of ``block``
    weights (row-major; ``W.numel()`` must be a multiple of ``block``) and
    return the codeword tensor of the same shape, differentiable in W and the
    codebook."""
    if W.numel() % block:
        raise ValueError(f"W.numel() = {W.numel()} is not a multiple of block = {block}")
    out = BcjrQuant.apply(W.reshape(-1, block), codebook, state_bits, k, T, hard)
    return out.reshape(W.shape)

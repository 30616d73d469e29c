"""Annealed quantisation-aware training of one weight matrix.

The loop of the paper's Algorithm "BCJR-QAT" (Sec. 3.7) for one layer, with
the exponential temperature schedule of Sec. 3.6 (Eq. anneal): at every step
the soft codeword of the current pre-image W is taken at temperature T_t,
a reconstruction loss is evaluated on it, its gradient is pulled back
through the soft codeword by the library's VJP, and an optimiser step moves
W.  At the end W is snapped to its Viterbi codeword.

Options beyond the paper's runs, each named there:
  * codebook learning: the VJP's dCodebook also moves the codebook (the
    paper's limitations section notes the relaxation admits it);
  * BCJR-STE: the forward value is the Viterbi codeword and the backward
    pass the temperature-T VJP (Sec. "BCJR-STE variant");
  * the drift-budget feasibility check of the paper's appendix: the
    expected nearest-codeword distance r = sigma_w / sqrt(2 pi S) against
    the largest drift lr * N * g_max that clipped gradient steps allow.

The loss is ||W_hat - W_target||_F^2, or with a proxy Hessian H = X^T X / n
of layer inputs X the layer-output error tr((W_hat - W_t) H (W_hat - W_t)^T).
Every trellis computation and every optimiser update runs in the library's
HIP kernels; the loss residual and the product with H are plain tensor
operations on the device.
"""
from __future__ import annotations

import dataclasses
import math

import torch

from . import (bcjr_soft_codeword, bcjr_soft_codeword_vjp, bcjr_ste_vjp, bcjr_vec_soft_codeword,
               bcjr_vec_soft_codeword_vjp, bcjr_vec_viterbi_decode, qat_adam_step, qat_sgd_step,
               viterbi_decode)

__all__ = ["QATConfig", "QATResult", "anneal_temperatures", "drift_budget", "anneal_qat"]


def anneal_temperatures(T0: float, T_end: float, steps: int):
    """T_i = T0 (T_end / T0)^(i / (steps - 1)), i = 0 .. steps - 1 (Eq. anneal,
    sampled at both ends)."""
    if steps < 1:
        raise ValueError("steps >= 1")
    if steps == 1:
        return [float(T0)]
    return [float(T0 * (T_end / T0) ** (i / (steps - 1))) for i in range(steps)]


def drift_budget(sigma_w: float, S: int, lr: float, steps: int, g_max: float) -> dict:
    """Necessary condition for leaving the initial Viterbi basin (the paper's
    drift-budget appendix): the per-element nearest-codeword distance
    r = sigma_w / sqrt(2 pi S) must be below the largest latent drift
    lr * steps * g_max reachable with gradients clipped at g_max."""
    r = sigma_w / math.sqrt(2.0 * math.pi * S)
    bound = lr * steps * g_max
    return {"r_voronoi": r, "max_drift": bound, "escape_possible": bound > r}


@dataclasses.dataclass
class QATConfig:
    state_bits: int
    k: int
    V: int = 1                   # weights per trellis step (1 or 2)
    block: int = 256             # weights per trellis block
    T0: float = 0.1
    T_end: float = 1e-3
    steps: int = 8
    lr: float = 1e-3
    grad_clip: float = 1.0       # elementwise clip of the pre-image gradient (g_max)
    optimizer: str = "adam"      # "adam" or "sgd"
    betas: tuple = (0.9, 0.999)
    eps: float = 1e-8
    learn_codebook: bool = False
    lr_codebook: float = 1e-4
    ste: bool = False


@dataclasses.dataclass
class QATResult:
    W: torch.Tensor              # final pre-image
    codebook: torch.Tensor       # final codebook
    W_hard: torch.Tensor         # Viterbi codeword of W
    temps: list
    losses: list                 # loss of each step's forward value
    loss_hard: float             # loss of W_hard
    loss_ptq: float              # loss of the Viterbi codeword of the initial W
    max_drift: float             # max |W - W_init| reached
    budget: dict                 # drift_budget() of the run's settings


def _loss_and_grad(W_hat, target, H):
    R = W_hat - target
    if H is None:
        return float((R * R).sum()), 2.0 * R
    RH = R @ H
    return float((RH * R).sum()), 2.0 * RH


def anneal_qat(W_init, codebook, cfg: QATConfig, target=None, H=None, stream=None) -> QATResult:
    """Run cfg.steps annealed steps on a [rows, cols] float32 device tensor.

    W_init is the starting pre-image (e.g. the weights themselves or a PTQ
    solution); target (default W_init) is what the codeword should
    reconstruct; H is an optional [cols, cols] proxy Hessian.  codebook is
    [S] (V = 1) or [S, V]; it is copied, and learned when
    cfg.learn_codebook.
    """
    n, k, V, blk = cfg.state_bits, cfg.k, cfg.V, cfg.block
    if W_init.dim() != 2 or W_init.numel() % blk:
        raise ValueError("W_init must be [rows, cols] with rows * cols a multiple of block")
    if cfg.optimizer not in ("adam", "sgd"):
        raise ValueError("optimizer must be 'adam' or 'sgd'")
    target = W_init if target is None else target
    W = W_init.detach().clone().contiguous()
    c = codebook.detach().clone().contiguous()
    mW, vW = torch.zeros_like(W), torch.zeros_like(W)
    mc, vc = torch.zeros_like(c), torch.zeros_like(c)
    temps = anneal_temperatures(cfg.T0, cfg.T_end, cfg.steps)
    b1, b2 = cfg.betas

    def forward(Wb, T):
        if cfg.ste:
            if V == 1:
                return viterbi_decode(Wb, c, n, k, stream=stream)[1]
            return bcjr_vec_viterbi_decode(Wb, c, n, k, V, stream=stream)[1]
        if V == 1:
            return bcjr_soft_codeword(Wb, c, n, k, T, want_logZ=False, stream=stream)[0]
        return bcjr_vec_soft_codeword(Wb, c, n, k, V, T, want_logZ=False, stream=stream)[0]

    def backward(Wb, T, G, fwd):
        want_dc = cfg.learn_codebook
        if V == 1:
            if cfg.ste:
                return bcjr_ste_vjp(Wb, c, n, k, T, fwd, G, want_dCodebook=want_dc, stream=stream)
            return bcjr_soft_codeword_vjp(Wb, c, n, k, T, G, want_dCodebook=want_dc, stream=stream)
        return bcjr_vec_soft_codeword_vjp(Wb, c, n, k, V, T, G, want_dCodebook=want_dc,
                                          stream=stream)

    losses = []
    for i, T in enumerate(temps):
        Wb = W.view(-1, blk)
        fwd = forward(Wb, T)
        loss, G = _loss_and_grad(fwd.view_as(W), target, H)
        losses.append(loss)
        dW, dc = backward(Wb, T, G.contiguous().view(-1, blk), fwd)
        if cfg.optimizer == "adam":
            qat_adam_step(W.view(-1, blk), dW, mW.view(-1, blk), vW.view(-1, blk), cfg.lr, b1, b2,
                          cfg.eps, i + 1, cfg.grad_clip, stream=stream)
            if cfg.learn_codebook:
                qat_adam_step(c, dc, mc, vc, cfg.lr_codebook, b1, b2, cfg.eps, i + 1, 0.0,
                              stream=stream)
        else:
            qat_sgd_step(W.view(-1, blk), dW, cfg.lr, cfg.grad_clip, stream=stream)
            if cfg.learn_codebook:
                qat_sgd_step(c, dc, cfg.lr_codebook, 0.0, stream=stream)

    def snap(Wm, cb):
        Wb = Wm.contiguous().view(-1, blk)
        if V == 1:
            return viterbi_decode(Wb, cb, n, k, stream=stream)[1].view_as(Wm)
        return bcjr_vec_viterbi_decode(Wb, cb, n, k, V, stream=stream)[1].view_as(Wm)

    W_hard = snap(W, c)
    loss_hard = _loss_and_grad(W_hard, target, H)[0]
    # the PTQ reference: the initial weights snapped with the initial codebook
    loss_ptq = _loss_and_grad(snap(W_init.detach(), codebook.detach().contiguous()), target, H)[0]
    sigma = float(target.float().std())
    return QATResult(W=W, codebook=c, W_hard=W_hard, temps=temps, losses=losses,
                     loss_hard=loss_hard, loss_ptq=loss_ptq,
                     max_drift=float((W - W_init).abs().max()),
                     budget=drift_budget(sigma, 1 << n, cfg.lr, cfg.steps, cfg.grad_clip))

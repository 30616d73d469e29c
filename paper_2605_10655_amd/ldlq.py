"""Hessian-weighted trellis rounding: BlockLDLQ with the Viterbi quantiser.

The PTQ reference of the paper's oracle-bound appendix is the minimiser of
the Hessian-weighted reconstruction loss
    L_HW(W_hat) = 1/2 tr((W - W_hat) H (W - W_hat)^T)          (Eq. LHW)
over the trellis codewords, reached QTIP-style by BlockLDLQ (Eq. WPTQ).  The
weights are [rows, cols]; H is the [cols, cols] proxy Hessian of the layer
inputs; each row is cut into trellis blocks of `block` consecutive columns.

Factor H = M D M^T with M unit block-upper-triangular and D block-diagonal
(blocks of `block` columns).  Then for one row with error e = w - w_hat,
    e H e^T = sum_k (e M)_k D_k (e M)_k^T,   (e M)_k = e_k + sum_{j<k} e_j M_jk,
so the column blocks are rounded in order, block k to the trellis codeword
nearest to the target
    t_k = w_k + sum_{j<k} (w_j - w_hat_j) M_jk,
which makes (e M)_k the block's own rounding error.  Each block's rounding is
one batched `viterbi_decode` over the rows (exact minimum-distortion path of
the target; D_k's off-diagonal coupling inside a block is not modelled, as
in QTIP).  The factorisation and the feedback products are library linear
algebra (Cholesky, triangular solves, GEMMs) on the device; every trellis
decode runs in the library's Viterbi kernel.
"""
from __future__ import annotations

import torch

from . import bcjr_vec_viterbi_decode, viterbi_decode

__all__ = ["block_ldl", "ldlq_viterbi", "hw_loss"]


def block_ldl(H: torch.Tensor, block: int):
    """H = M D M^T, M unit block-upper-triangular, D block-diagonal.

    From the upper Cholesky factor H = R R^T (R upper triangular, the
    Cholesky factor of H with the index order reversed): M = R B^{-1} and
    D = B B^T with B = blockdiag(R_kk)."""
    d = H.shape[0]
    if H.shape != (d, d) or d % block:
        raise ValueError("H must be square with a size that is a multiple of block")
    Hr = torch.flip(H, (0, 1))
    C = torch.linalg.cholesky(Hr)                     # Hr = C C^T, C lower
    R = torch.flip(C, (0, 1))                         # H = R R^T, R upper
    M = torch.zeros_like(R)
    D = torch.zeros_like(R)
    eye = torch.eye(block, dtype=H.dtype, device=H.device)
    for k in range(0, d, block):
        Rkk = R[k:k + block, k:k + block]
        Rinv = torch.linalg.solve_triangular(Rkk, eye, upper=True)
        M[:, k:k + block] = R[:, k:k + block] @ Rinv
        D[k:k + block, k:k + block] = Rkk @ Rkk.T
    return M, D


def hw_loss(W, W_hat, H) -> float:
    """1/2 tr((W - W_hat) H (W - W_hat)^T)  (Eq. LHW)."""
    E = (W - W_hat).double()
    return 0.5 * float(((E @ H.double()) * E).sum())


def ldlq_viterbi(W, codebook, state_bits: int, k: int, H, block: int = 256, V: int = 1,
                 damp: float = 0.01, return_targets: bool = False, stream=None):
    """BlockLDLQ rounding of W [rows, cols] (float32, device) to trellis
    codewords.  H [cols, cols] is damped by damp * mean(diag H) on the
    diagonal before factorisation (the usual regularisation of a sample
    Hessian).  Returns (W_hat [rows, cols], states [cols // block, rows,
    block // V]) and, with return_targets, the per-block targets t_k."""
    rows, cols = W.shape
    if cols % block or block % V:
        raise ValueError("cols must be a multiple of block, block a multiple of V")
    Hd = H.double()
    Hd = Hd + damp * Hd.diagonal().mean() * torch.eye(cols, dtype=Hd.dtype, device=Hd.device)
    M, _ = block_ldl(Hd, block)
    Mf = M.float()
    W = W.contiguous()
    W_hat = torch.empty_like(W)
    Err = torch.zeros_like(W)
    nb = cols // block
    states = torch.empty((nb, rows, block // V), dtype=torch.int32, device=W.device)
    targets = torch.empty((nb, rows, block), dtype=W.dtype, device=W.device) if return_targets else None
    for kb in range(nb):
        sl = slice(kb * block, (kb + 1) * block)
        t = W[:, sl]
        if kb > 0:
            t = t + Err[:, :kb * block] @ Mf[:kb * block, sl]
        t = t.contiguous()
        if return_targets:
            targets[kb] = t
        if V == 1:
            _, wh = viterbi_decode(t, codebook, state_bits, k, states=states[kb], stream=stream)
        else:
            _, wh = bcjr_vec_viterbi_decode(t, codebook, state_bits, k, V, states=states[kb],
                                            stream=stream)
        W_hat[:, sl] = wh
        Err[:, sl] = W[:, sl] - wh
    return (W_hat, states, targets) if return_targets else (W_hat, states)

"""Hessian-weighted trellis rounding: BlockLDLQ with the Viterbi quantiser.

The PTQ reference of the paper's oracle-bound appendix is the minimiser of
the Hessian-weighted reconstruction loss
    L_HW(W_hat) = 1/2 tr((W - W_hat) H (W - W_hat)^T)          (Eq. LHW)
over the trellis codewords, reached QTIP-style by BlockLDLQ (Eq. WPTQ).  The
weights are [rows, cols]; H is the [cols, cols] proxy Hessian of the layer
inputs; each row is cut into trellis blocks of `block` consecutive columns.

With H = M D M^T (M unit block-upper-triangular, D block-diagonal), one
row's error e = w - w_hat gives e H e^T = sum_k (e M)_k D_k (e M)_k^T with
(e M)_k = e_k + sum_{j<k} e_j M_jk, so the column blocks are rounded in
order, block k to the codeword nearest to its target
    t_k = w_k + sum_{j<k} (w_j - w_hat_j) M_jk.

This module only marshals tensors for the library's C ABI: the damping, the
factorisation, the feedback products and every decode run in HIP kernels
(bcjr_block_ldl, bcjr_ldlq_viterbi).  ``hw_loss`` is an evaluation helper
for reports and tests, not part of the rounding.
"""
from __future__ import annotations

import ctypes

import torch

from . import _check_in, _ptr, _raise, _stream, load_library

__all__ = ["block_ldl", "ldlq_viterbi", "hw_loss"]


def _lib():
    L = load_library()
    if not getattr(L, "_ldlq_bound", False):
        vp, i64, ci, cd, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_size_t
        L.bcjr_block_ldl_workspace_bytes.argtypes = [i64, i64]
        L.bcjr_block_ldl_workspace_bytes.restype = sz
        L.bcjr_block_ldl.argtypes = [vp, i64, i64, cd, vp, vp, vp, sz, vp]
        L.bcjr_block_ldl.restype = ci
        L.bcjr_ldlq_workspace_bytes.argtypes = [i64, i64, i64, ci, ci, ci]
        L.bcjr_ldlq_workspace_bytes.restype = sz
        L.bcjr_ldlq_viterbi.argtypes = [vp, i64, i64, vp, ci, ci, ci, vp, i64, cd, vp, vp, vp, vp, sz,
                                        vp]
        L.bcjr_ldlq_viterbi.restype = ci
        L._ldlq_bound = True
    return L


def block_ldl(H: torch.Tensor, block: int, damp: float = 0.0, want_D: bool = True, stream=None):
    """(H + damp mean(diag H) I) = M D M^T on the device: M unit
    block-upper-triangular, D block-diagonal, both [d, d] float64."""
    lib = _lib()
    d = H.shape[0]
    if H.dim() != 2 or H.shape != (d, d) or d % block:
        raise ValueError("H must be square with a size that is a multiple of block")
    _check_in("H", H)
    M = torch.empty((d, d), dtype=torch.float64, device=H.device)
    D = torch.empty((d, d), dtype=torch.float64, device=H.device) if want_D else None
    nbytes = lib.bcjr_block_ldl_workspace_bytes(d, block)
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=H.device)
    rc = lib.bcjr_block_ldl(_ptr(H), d, block, float(damp), _ptr(M), _ptr(D), _ptr(ws), ws.numel(),
                            _stream(stream))
    _raise("bcjr_block_ldl", rc)
    return M, D


def hw_loss(W, W_hat, H) -> float:
    """1/2 tr((W - W_hat) H (W - W_hat)^T)  (Eq. LHW), in float64."""
    E = (W - W_hat).double()
    return 0.5 * float(((E @ H.double()) * E).sum())


def ldlq_viterbi(W, codebook, state_bits: int, k: int, H, block: int = 256, V: int = 1,
                 damp: float = 0.01, return_targets: bool = False, stream=None):
    """BlockLDLQ rounding of W [rows, cols] (float32, device) to trellis
    codewords.  H [cols, cols] (float32) is damped by damp * mean(diag H) on
    the diagonal before factorisation.  Returns (W_hat [rows, cols], states
    [cols // block, rows, block // V]) and, with return_targets, the
    per-block targets t_k [cols // block, rows, block]."""
    lib = _lib()
    rows, cols = W.shape
    if cols % block or block % V:
        raise ValueError("cols must be a multiple of block, block a multiple of V")
    _check_in("W", W)
    dev = W.device
    _check_in("H", H, (cols, cols), device=dev)
    _check_in("codebook", codebook, device=dev)
    if codebook.numel() != (1 << state_bits) * V:
        raise ValueError("codebook must hold 2^state_bits x V values")
    nb = cols // block
    W_hat = torch.empty_like(W)
    states = torch.empty((nb, rows, block // V), dtype=torch.int32, device=dev)
    targets = torch.empty((nb, rows, block), dtype=W.dtype, device=dev) if return_targets else None
    nbytes = lib.bcjr_ldlq_workspace_bytes(rows, cols, block, state_bits, k, V)
    if nbytes == 0:
        raise ValueError("unsupported shape for the BlockLDLQ decode")
    ws = torch.empty(int(nbytes), dtype=torch.uint8, device=dev)
    rc = lib.bcjr_ldlq_viterbi(_ptr(W), rows, cols, _ptr(codebook), state_bits, k, V, _ptr(H), block,
                               float(damp), _ptr(W_hat), _ptr(states), _ptr(targets), _ptr(ws),
                               ws.numel(), _stream(stream))
    _raise("bcjr_ldlq_viterbi", rc)
    return (W_hat, states, targets) if return_targets else (W_hat, states)

"""MI355X (gfx950) BCJR soft-codeword library: Python binding.

Thin ctypes marshalling over the C ABI declared in ``include/bcjr.h``
(``libbcjr.so``, built in-tree by ``build.py``).  Every step of the
computation runs in the library's HIP kernels; this module only checks
tensor shapes, allocates outputs and the workspace through PyTorch, and
passes raw device pointers and the current HIP stream.

The autograd layer (``BcjrQuant``, soft or BCJR-STE forward) is in
``paper_2605_10655_amd.autograd``.

Functions keep the C names:
    bcjr_soft_codeword(w, codebook, state_bits, k, T)            -> (w_soft, logZ)
    bcjr_soft_codeword_vjp(w, codebook, state_bits, k, T, g)     -> (dW, dCodebook)
    bcjr_soft_codeword_fwd_vjp(w, codebook, state_bits, k, T, g) -> (w_soft, logZ, dW, dCodebook)
    bcjr_soft_codeword_fwd_vjp_noalloc(w, codebook, state_bits, k, T, g, w_soft=..., ...)
    bcjr_ste_vjp(w, codebook, state_bits, k, T, w_hard, g)       -> (dW, dCodebook)
    viterbi_decode(w, codebook, state_bits, k)                   -> (states, w_hard)
    bcjr_workspace_bytes(B, L, state_bits, k, op)                -> int
and the vector-emission forms (V weights per step, codebook [S, V]):
    bcjr_vec_soft_codeword(w, codebook, state_bits, k, V, T)          -> (w_soft, logZ)
    bcjr_vec_soft_codeword_vjp(w, codebook, state_bits, k, V, T, g)   -> (dW, dCodebook)
    bcjr_vec_soft_codeword_fwd_vjp(w, codebook, state_bits, k, V, T, g)
    bcjr_vec_viterbi_decode(w, codebook, state_bits, k, V)            -> (states, w_hard)
    bcjr_vec_workspace_bytes(B, L, state_bits, k, V, op)              -> int
and the training helpers:
    bcjr_gaussian_codebook(state_bits, V, seed)                       -> codebook [S] or [S, V]
    qat_adam_step(param, grad, m, v, lr, beta1, beta2, eps, step, grad_clip)   (in place)
    qat_sgd_step(param, grad, lr, grad_clip)                          (in place)
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "BcjrError", "OP_FWD", "OP_VJP", "OP_FWD_VJP", "OP_VITERBI", "library_path", "load_library",
    "bcjr_workspace_bytes", "bcjr_status_string", "bcjr_soft_codeword", "bcjr_soft_codeword_vjp",
    "bcjr_soft_codeword_fwd_vjp", "bcjr_soft_codeword_fwd_vjp_noalloc", "bcjr_ste_vjp",
    "viterbi_decode", "bcjr_vec_workspace_bytes",
    "bcjr_vec_soft_codeword", "bcjr_vec_soft_codeword_vjp", "bcjr_vec_soft_codeword_fwd_vjp",
    "bcjr_vec_viterbi_decode", "bcjr_gaussian_codebook", "qat_adam_step", "qat_sgd_step",
]

OP_FWD, OP_VJP, OP_FWD_VJP, OP_VITERBI = 0, 1, 2, 3
STATUS = {0: "BCJR_OK", -1: "BCJR_ERR_INVALID_ARG", -2: "BCJR_ERR_UNSUPPORTED",
          -3: "BCJR_ERR_WORKSPACE", -4: "BCJR_ERR_HIP"}

_HERE = os.path.dirname(os.path.abspath(__file__))
_lib = None


class BcjrError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} returned {STATUS.get(status, status)}: {bcjr_status_string(status)}")


def library_path() -> str:
    return os.path.join(_HERE, "libbcjr.so")


def load_library():
    """Load libbcjr.so.  Raises ImportError if it was not built: there is no
    fallback implementation."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2605_10655_amd.build`")
    L = ctypes.CDLL(path)
    vp, i64, ci, cf, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.bcjr_workspace_bytes.argtypes = [i64, i64, ci, ci, ci]
    L.bcjr_workspace_bytes.restype = sz
    L.bcjr_status_string.argtypes = [ci]
    L.bcjr_status_string.restype = ctypes.c_char_p
    L.bcjr_soft_codeword.argtypes = [vp, i64, i64, vp, ci, ci, cf, vp, vp, vp, sz, vp]
    L.bcjr_soft_codeword_vjp.argtypes = [vp, i64, i64, vp, ci, ci, cf, vp, vp, vp, vp, sz, vp]
    L.bcjr_soft_codeword_fwd_vjp.argtypes = [vp, i64, i64, vp, ci, ci, cf, vp, vp, vp, vp, vp, vp,
                                             sz, vp]
    L.bcjr_soft_codeword_fwd_vjp_noalloc.argtypes = [vp, i64, i64, vp, ci, ci, cf, vp, vp, vp, vp,
                                                     vp, vp]
    L.bcjr_ste_vjp.argtypes = [vp, i64, i64, vp, ci, ci, cf, vp, vp, vp, vp, vp, sz, vp]
    L.viterbi_decode.argtypes = [vp, i64, i64, vp, ci, ci, vp, vp, vp, sz, vp]
    L.bcjr_vec_workspace_bytes.argtypes = [i64, i64, ci, ci, ci, ci]
    L.bcjr_vec_workspace_bytes.restype = sz
    L.bcjr_vec_soft_codeword.argtypes = [vp, i64, i64, vp, ci, ci, ci, cf, vp, vp, vp, sz, vp]
    L.bcjr_vec_soft_codeword_vjp.argtypes = [vp, i64, i64, vp, ci, ci, ci, cf, vp, vp, vp, vp, sz,
                                             vp]
    L.bcjr_vec_soft_codeword_fwd_vjp.argtypes = [vp, i64, i64, vp, ci, ci, ci, cf, vp, vp, vp, vp,
                                                 vp, vp, sz, vp]
    L.bcjr_vec_viterbi_decode.argtypes = [vp, i64, i64, vp, ci, ci, ci, vp, vp, vp, sz, vp]
    u64 = ctypes.c_uint64
    L.bcjr_gaussian_codebook.argtypes = [vp, ci, ci, u64, vp]
    L.qat_adam_step.argtypes = [vp, vp, vp, vp, i64, cf, cf, cf, cf, i64, cf, vp]
    L.qat_sgd_step.argtypes = [vp, vp, i64, cf, cf, vp]
    for f in (L.bcjr_soft_codeword, L.bcjr_soft_codeword_vjp, L.bcjr_soft_codeword_fwd_vjp,
              L.bcjr_soft_codeword_fwd_vjp_noalloc, L.bcjr_ste_vjp, L.viterbi_decode,
              L.bcjr_vec_soft_codeword,
              L.bcjr_vec_soft_codeword_vjp, L.bcjr_vec_soft_codeword_fwd_vjp,
              L.bcjr_vec_viterbi_decode, L.bcjr_gaussian_codebook, L.qat_adam_step,
              L.qat_sgd_step):
        f.restype = ci
    _lib = L
    return L


def bcjr_workspace_bytes(B: int, L: int, state_bits: int, k: int, op: int) -> int:
    return int(load_library().bcjr_workspace_bytes(B, L, state_bits, k, op))


def bcjr_status_string(status: int) -> str:
    return load_library().bcjr_status_string(status).decode()


# ---------------------------------------------------------------- helpers
def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check_in(name, t, shape=None, dtype=None, device=None):
    """Every tensor handed to the library, input or caller-supplied output:
    a contiguous device tensor of the expected dtype, shape and device (the
    kernels index it as a dense array of exactly that size)."""
    torch = _torch()
    dtype = dtype or torch.float32
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the call's tensors on {device}")


def _check_out(name, t, shape, device, dtype=None):
    if t is not None:
        _check_in(name, t, shape, dtype, device)


def _keep_alive(stream, *tensors):
    """Tensors this module allocated come from PyTorch's caching allocator on
    the current stream; when the launch went to another stream, tell the
    allocator so that their memory is not handed out again while the
    kernels may still use it."""
    if stream is None:
        return
    torch = _torch()
    if stream == torch.cuda.current_stream(stream.device):
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def _ws_bytes(ws):
    return ws.numel() * ws.element_size()


def _check_ws(ws, device):
    torch = _torch()
    if not isinstance(ws, torch.Tensor) or not ws.is_cuda:
        raise TypeError("workspace must be a CUDA (HIP) tensor")
    if not ws.is_contiguous():
        raise ValueError("workspace must be contiguous")
    if ws.device != device:
        raise ValueError(f"workspace is on {ws.device}, the call's tensors on {device}")


def _workspace(workspace, B, L, state_bits, k, op, device):
    torch = _torch()
    if workspace is not None:
        _check_ws(workspace, device)
        return workspace
    nbytes = bcjr_workspace_bytes(B, L, state_bits, k, op)
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def _shape(w):
    if w.dim() != 2:
        raise ValueError("w must be [B, L]")
    return int(w.shape[0]), int(w.shape[1])


def _raise(fn, rc):
    if rc != 0:
        raise BcjrError(fn, rc)


# ---------------------------------------------------------------- API
def bcjr_soft_codeword(w, codebook, state_bits, k, T, *, w_soft=None, logZ=None, want_logZ=True,
                       workspace=None, stream=None):
    """Soft codeword w_soft[B, L] and natural-log partition function logZ[B]."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _check_in("codebook", codebook, (1 << state_bits,), device=dev)
    _check_out("w_soft", w_soft, (B, L), dev)
    _check_out("logZ", logZ, (B,), dev)
    if w_soft is None:
        w_soft = torch.empty_like(w)
    if logZ is None and want_logZ:
        logZ = torch.empty(B, dtype=torch.float32, device=dev)
    ws = _workspace(workspace, B, L, state_bits, k, OP_FWD, dev)
    rc = lib.bcjr_soft_codeword(_ptr(w), B, L, _ptr(codebook), state_bits, k, float(T),
                                _ptr(w_soft), _ptr(logZ), _ptr(ws), _ws_bytes(ws), _stream(stream))
    _raise("bcjr_soft_codeword", rc)
    _keep_alive(stream, w_soft, logZ, ws)
    return w_soft, logZ


def bcjr_soft_codeword_vjp(w, codebook, state_bits, k, T, grad_w_soft, *, want_dW=True,
                           want_dCodebook=True, dW=None, dCodebook=None, workspace=None,
                           stream=None):
    """VJP of <grad_w_soft, w_soft>: (dW[B, L] or None, dCodebook[S] or None)."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _check_in("codebook", codebook, (1 << state_bits,), device=dev)
    _check_in("grad_w_soft", grad_w_soft, (B, L), device=dev)
    _check_out("dW", dW, (B, L), dev)
    _check_out("dCodebook", dCodebook, (1 << state_bits,), dev)
    if dW is None and want_dW:
        dW = torch.empty_like(w)
    if dCodebook is None and want_dCodebook:
        dCodebook = torch.empty(1 << state_bits, dtype=torch.float32, device=dev)
    ws = _workspace(workspace, B, L, state_bits, k, OP_VJP, dev)
    rc = lib.bcjr_soft_codeword_vjp(_ptr(w), B, L, _ptr(codebook), state_bits, k, float(T),
                                    _ptr(grad_w_soft), _ptr(dW), _ptr(dCodebook), _ptr(ws),
                                    _ws_bytes(ws), _stream(stream))
    _raise("bcjr_soft_codeword_vjp", rc)
    _keep_alive(stream, dW, dCodebook, ws)
    return dW, dCodebook


def bcjr_soft_codeword_fwd_vjp(w, codebook, state_bits, k, T, grad_w_soft, *, want_w_soft=True,
                               want_logZ=True, want_dW=True, want_dCodebook=True, w_soft=None,
                               logZ=None, dW=None, dCodebook=None, workspace=None, stream=None):
    """Forward outputs and the VJP in one call: (w_soft, logZ, dW, dCodebook)."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _check_in("codebook", codebook, (1 << state_bits,), device=dev)
    _check_in("grad_w_soft", grad_w_soft, (B, L), device=dev)
    for name, t, shp in (("w_soft", w_soft, (B, L)), ("logZ", logZ, (B,)), ("dW", dW, (B, L)),
                         ("dCodebook", dCodebook, (1 << state_bits,))):
        _check_out(name, t, shp, dev)
    if w_soft is None and want_w_soft:
        w_soft = torch.empty_like(w)
    if logZ is None and want_logZ:
        logZ = torch.empty(B, dtype=torch.float32, device=dev)
    if dW is None and want_dW:
        dW = torch.empty_like(w)
    if dCodebook is None and want_dCodebook:
        dCodebook = torch.empty(1 << state_bits, dtype=torch.float32, device=dev)
    ws = _workspace(workspace, B, L, state_bits, k, OP_FWD_VJP, dev)
    rc = lib.bcjr_soft_codeword_fwd_vjp(_ptr(w), B, L, _ptr(codebook), state_bits, k, float(T),
                                        _ptr(grad_w_soft), _ptr(w_soft), _ptr(logZ), _ptr(dW),
                                        _ptr(dCodebook), _ptr(ws), _ws_bytes(ws), _stream(stream))
    _raise("bcjr_soft_codeword_fwd_vjp", rc)
    _keep_alive(stream, w_soft, logZ, dW, dCodebook, ws)
    return w_soft, logZ, dW, dCodebook


def bcjr_soft_codeword_fwd_vjp_noalloc(w, codebook, state_bits, k, T, grad_w_soft, *, w_soft,
                                       logZ=None, dW=None, dCodebook=None, stream=None):
    """bcjr_soft_codeword_fwd_vjp on the library's static per-GPU scratch
    array: no workspace, and every output is the caller's (nothing is
    allocated here either).  Returns (w_soft, logZ, dW, dCodebook)."""
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _check_in("codebook", codebook, (1 << state_bits,), device=dev)
    _check_in("grad_w_soft", grad_w_soft, (B, L), device=dev)
    for name, t, shp in (("w_soft", w_soft, (B, L)), ("logZ", logZ, (B,)), ("dW", dW, (B, L)),
                         ("dCodebook", dCodebook, (1 << state_bits,))):
        _check_out(name, t, shp, dev)
    rc = lib.bcjr_soft_codeword_fwd_vjp_noalloc(_ptr(w), B, L, _ptr(codebook), state_bits, k,
                                                float(T), _ptr(grad_w_soft), _ptr(w_soft),
                                                _ptr(logZ), _ptr(dW), _ptr(dCodebook),
                                                _stream(stream))
    _raise("bcjr_soft_codeword_fwd_vjp_noalloc", rc)
    return w_soft, logZ, dW, dCodebook


def bcjr_ste_vjp(w, codebook, state_bits, k, T, w_hard, grad_w_soft, *, want_dW=True,
                 want_dCodebook=True, dW=None, dCodebook=None, workspace=None, stream=None):
    """Backward pass of BCJR-STE: the VJP of <grad_w_soft, w_soft> at temperature T,
    given the forward pass's Viterbi codewords w_hard[B, L] (the centring
    reference of the low-temperature variant).  (dW or None, dCodebook or None)."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _check_in("codebook", codebook, (1 << state_bits,), device=dev)
    _check_in("w_hard", w_hard, (B, L), device=dev)
    _check_in("grad_w_soft", grad_w_soft, (B, L), device=dev)
    _check_out("dW", dW, (B, L), dev)
    _check_out("dCodebook", dCodebook, (1 << state_bits,), dev)
    if dW is None and want_dW:
        dW = torch.empty_like(w)
    if dCodebook is None and want_dCodebook:
        dCodebook = torch.empty(1 << state_bits, dtype=torch.float32, device=dev)
    ws = _workspace(workspace, B, L, state_bits, k, OP_VJP, dev)
    rc = lib.bcjr_ste_vjp(_ptr(w), B, L, _ptr(codebook), state_bits, k, float(T), _ptr(w_hard),
                          _ptr(grad_w_soft), _ptr(dW), _ptr(dCodebook), _ptr(ws), _ws_bytes(ws),
                          _stream(stream))
    _raise("bcjr_ste_vjp", rc)
    _keep_alive(stream, dW, dCodebook, ws)
    return dW, dCodebook


def viterbi_decode(w, codebook, state_bits, k, *, want_w_hard=True, states=None, w_hard=None,
                   workspace=None, stream=None):
    """Minimum-distortion path: (states[B, L] int32, w_hard[B, L] or None)."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _check_in("codebook", codebook, (1 << state_bits,), device=dev)
    _check_out("states", states, (B, L), dev, torch.int32)
    _check_out("w_hard", w_hard, (B, L), dev)
    if states is None:
        states = torch.empty((B, L), dtype=torch.int32, device=dev)
    if w_hard is None and want_w_hard:
        w_hard = torch.empty_like(w)
    ws = _workspace(workspace, B, L, state_bits, k, OP_VITERBI, dev)
    rc = lib.viterbi_decode(_ptr(w), B, L, _ptr(codebook), state_bits, k, _ptr(states),
                            _ptr(w_hard), _ptr(ws), _ws_bytes(ws), _stream(stream))
    _raise("viterbi_decode", rc)
    _keep_alive(stream, states, w_hard, ws)
    return states, w_hard


# ---------------------------------------------------------------- vector emission
def bcjr_vec_workspace_bytes(B: int, L: int, state_bits: int, k: int, V: int, op: int) -> int:
    return int(load_library().bcjr_vec_workspace_bytes(B, L, state_bits, k, V, op))


def _vec_codebook(codebook, state_bits, V, device, name="codebook"):
    S = 1 << state_bits
    _check_in(name, codebook, device=device)
    if codebook.numel() != S * V:
        raise ValueError(f"{name} must hold {S} x {V} values, got {tuple(codebook.shape)}")


def _vec_workspace(workspace, B, L, state_bits, k, V, op, device):
    torch = _torch()
    if workspace is not None:
        _check_ws(workspace, device)
        return workspace
    nbytes = bcjr_vec_workspace_bytes(B, L, state_bits, k, V, op)
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def bcjr_vec_soft_codeword(w, codebook, state_bits, k, V, T, *, w_soft=None, logZ=None,
                           want_logZ=True, workspace=None, stream=None):
    """Soft codeword w_soft[B, L] and logZ[B] with V weights per step."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _vec_codebook(codebook, state_bits, V, dev)
    _check_out("w_soft", w_soft, (B, L), dev)
    _check_out("logZ", logZ, (B,), dev)
    if w_soft is None:
        w_soft = torch.empty_like(w)
    if logZ is None and want_logZ:
        logZ = torch.empty(B, dtype=torch.float32, device=dev)
    ws = _vec_workspace(workspace, B, L, state_bits, k, V, OP_FWD, dev)
    rc = lib.bcjr_vec_soft_codeword(_ptr(w), B, L, _ptr(codebook), state_bits, k, V, float(T),
                                    _ptr(w_soft), _ptr(logZ), _ptr(ws), _ws_bytes(ws), _stream(stream))
    _raise("bcjr_vec_soft_codeword", rc)
    _keep_alive(stream, w_soft, logZ, ws)
    return w_soft, logZ


def bcjr_vec_soft_codeword_fwd_vjp(w, codebook, state_bits, k, V, T, grad_w_soft, *,
                                   want_w_soft=True, want_logZ=True, want_dW=True,
                                   want_dCodebook=True, w_soft=None, logZ=None, dW=None,
                                   dCodebook=None, workspace=None, stream=None):
    """(w_soft, logZ, dW, dCodebook) with V weights per step; dCodebook has
    the codebook's shape."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _vec_codebook(codebook, state_bits, V, dev)
    _check_in("grad_w_soft", grad_w_soft, (B, L), device=dev)
    for name, t, shp in (("w_soft", w_soft, (B, L)), ("logZ", logZ, (B,)), ("dW", dW, (B, L))):
        _check_out(name, t, shp, dev)
    if dCodebook is not None:
        _vec_codebook(dCodebook, state_bits, V, dev, "dCodebook")
    if w_soft is None and want_w_soft:
        w_soft = torch.empty_like(w)
    if logZ is None and want_logZ:
        logZ = torch.empty(B, dtype=torch.float32, device=dev)
    if dW is None and want_dW:
        dW = torch.empty_like(w)
    if dCodebook is None and want_dCodebook:
        dCodebook = torch.empty_like(codebook)
    ws = _vec_workspace(workspace, B, L, state_bits, k, V, OP_FWD_VJP, dev)
    rc = lib.bcjr_vec_soft_codeword_fwd_vjp(_ptr(w), B, L, _ptr(codebook), state_bits, k, V,
                                            float(T), _ptr(grad_w_soft), _ptr(w_soft), _ptr(logZ),
                                            _ptr(dW), _ptr(dCodebook), _ptr(ws), _ws_bytes(ws),
                                            _stream(stream))
    _raise("bcjr_vec_soft_codeword_fwd_vjp", rc)
    _keep_alive(stream, w_soft, logZ, dW, dCodebook, ws)
    return w_soft, logZ, dW, dCodebook


def bcjr_vec_soft_codeword_vjp(w, codebook, state_bits, k, V, T, grad_w_soft, *, want_dW=True,
                               want_dCodebook=True, dW=None, dCodebook=None, workspace=None,
                               stream=None):
    """(dW or None, dCodebook or None) with V weights per step."""
    out = bcjr_vec_soft_codeword_fwd_vjp(w, codebook, state_bits, k, V, T, grad_w_soft,
                                         want_w_soft=False, want_logZ=False, want_dW=want_dW,
                                         want_dCodebook=want_dCodebook, dW=dW, dCodebook=dCodebook,
                                         workspace=workspace, stream=stream)
    return out[2], out[3]


def bcjr_vec_viterbi_decode(w, codebook, state_bits, k, V, *, want_w_hard=True, states=None,
                            w_hard=None, workspace=None, stream=None):
    """(states[B, L // V] int32, w_hard[B, L] or None) with V weights per step."""
    torch = _torch()
    lib = load_library()
    B, L = _shape(w)
    _check_in("w", w)
    dev = w.device
    _vec_codebook(codebook, state_bits, V, dev)
    if L % V:
        raise ValueError(f"L = {L} is not a multiple of V = {V}")
    _check_out("states", states, (B, L // V), dev, torch.int32)
    _check_out("w_hard", w_hard, (B, L), dev)
    if states is None:
        states = torch.empty((B, L // V), dtype=torch.int32, device=dev)
    if w_hard is None and want_w_hard:
        w_hard = torch.empty_like(w)
    ws = _vec_workspace(workspace, B, L, state_bits, k, V, OP_VITERBI, dev)
    rc = lib.bcjr_vec_viterbi_decode(_ptr(w), B, L, _ptr(codebook), state_bits, k, V, _ptr(states),
                                     _ptr(w_hard), _ptr(ws), _ws_bytes(ws), _stream(stream))
    _raise("bcjr_vec_viterbi_decode", rc)
    _keep_alive(stream, states, w_hard, ws)
    return states, w_hard


# ---------------------------------------------------------------- training helpers
def bcjr_gaussian_codebook(state_bits, V=1, seed=0, *, out=None, device="cuda", stream=None):
    """Computed Gaussian codebook: [S] (V = 1) or [S, V] float32 on the device."""
    torch = _torch()
    lib = load_library()
    S = 1 << state_bits
    if out is None:
        out = torch.empty((S,) if V == 1 else (S, V), dtype=torch.float32, device=device)
    _check_in("out", out)
    if out.numel() != S * V:
        raise ValueError(f"out must hold {S} x {V} values")
    rc = lib.bcjr_gaussian_codebook(_ptr(out), state_bits, V, int(seed) & ((1 << 64) - 1),
                                    _stream(stream))
    _raise("bcjr_gaussian_codebook", rc)
    _keep_alive(stream, out)
    return out


def qat_adam_step(param, grad, m, v, lr, beta1=0.9, beta2=0.999, eps=1e-8, step=1, grad_clip=0.0,
                  stream=None):
    """One Adam step in place on param, m, v (same shape, float32, device)."""
    lib = load_library()
    for name, t in (("param", param), ("grad", grad), ("m", m), ("v", v)):
        _check_in(name, t, tuple(param.shape), device=param.device)
    rc = lib.qat_adam_step(_ptr(param), _ptr(grad), _ptr(m), _ptr(v), param.numel(), float(lr),
                           float(beta1), float(beta2), float(eps), int(step), float(grad_clip),
                           _stream(stream))
    _raise("qat_adam_step", rc)


def qat_sgd_step(param, grad, lr, grad_clip=0.0, stream=None):
    """param -= lr * clamp(grad, -grad_clip, grad_clip), in place."""
    lib = load_library()
    _check_in("param", param)
    _check_in("grad", grad, tuple(param.shape), device=param.device)
    rc = lib.qat_sgd_step(_ptr(param), _ptr(grad), param.numel(), float(lr), float(grad_clip),
                          _stream(stream))
    _raise("qat_sgd_step", rc)

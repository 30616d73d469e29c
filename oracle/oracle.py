"""ctypes binding of the plain fp64 CPU oracle (``bcjr_oracle.c``).

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
CPU-baseline leg of the benchmark may import this module.  It shares nothing
with the HIP implementation; inputs are converted exactly to float64 before
the call, so fp32 arrays reach the oracle unchanged.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bcjr_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build() -> str:
    """Compile the oracle with gcc (fp contraction off: the Viterbi metric
    rounds the product and the sum separately)."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-pthread", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        i64 = ctypes.c_int64
        ci = ctypes.c_int
        cd = ctypes.c_double
        L.oracle_soft_codeword.argtypes = [dp, i64, i64, dp, ci, ci, cd, dp, dp, ci]
        L.oracle_soft_codeword_vjp.argtypes = [dp, i64, i64, dp, ci, ci, cd, dp, dp, dp, dp, dp, ci]
        L.oracle_viterbi.argtypes = [dp, i64, i64, dp, ci, ci, ip, dp, ci]
        L.oracle_block_tables.argtypes = [dp, i64, dp, ci, ci, cd, dp, dp, dp, dp, dp]
        for f in (L.oracle_soft_codeword, L.oracle_soft_codeword_vjp, L.oracle_viterbi,
                  L.oracle_block_tables):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def _d(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a, ty=ctypes.c_double):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ty))


def _check(rc, name):
    if rc != 0:
        raise RuntimeError(f"{name} failed with status {rc}")


def soft_codeword(w, c, n, k, T, nthreads=None):
    """w[B, L] -> (w_soft[B, L] float64, logZ[B] float64)."""
    w = _d(w)
    c = _d(c)
    B, L = w.shape
    ws = np.empty((B, L), np.float64)
    lz = np.empty((B,), np.float64)
    rc = lib().oracle_soft_codeword(_ptr(w), B, L, _ptr(c), n, k, float(T), _ptr(ws),
                                    _ptr(lz), nthreads or default_threads())
    _check(rc, "oracle_soft_codeword")
    return ws, lz


def soft_codeword_vjp(w, c, n, k, T, g, want_dc=True, nthreads=None):
    """Returns (w_soft, logZ, dW, dc) in float64; dc is summed over blocks
    (None when want_dc is False)."""
    w = _d(w)
    c = _d(c)
    g = _d(g)
    B, L = w.shape
    assert g.shape == (B, L)
    ws = np.empty((B, L), np.float64)
    lz = np.empty((B,), np.float64)
    dW = np.empty((B, L), np.float64)
    dc = np.empty((1 << n,), np.float64) if want_dc else None
    rc = lib().oracle_soft_codeword_vjp(_ptr(w), B, L, _ptr(c), n, k, float(T), _ptr(g),
                                        _ptr(ws), _ptr(lz), _ptr(dW), _ptr(dc),
                                        nthreads or default_threads())
    _check(rc, "oracle_soft_codeword_vjp")
    return ws, lz, dW, dc


def viterbi(w, c, n, k, nthreads=None):
    """w[B, L] -> (states[B, L] int32, cost[B] float64)."""
    w = _d(w)
    c = _d(c)
    B, L = w.shape
    st = np.empty((B, L), np.int32)
    cost = np.empty((B,), np.float64)
    rc = lib().oracle_viterbi(_ptr(w), B, L, _ptr(c), n, k, _ptr(st, ctypes.c_int32),
                              _ptr(cost), nthreads or default_threads())
    _check(rc, "oracle_viterbi")
    return st, cost


def ste(w, c, n, k, T, g, want_dc=True, nthreads=None):
    """BCJR-STE (paper Sec. 3.5 and Sec. "BCJR-STE variant"): the forward
    output is the hard codeword c(s_t) of the minimum-distortion path
    (Sec. 3.2) and the backward pass is the VJP of the temperature-T soft
    codeword (Sec. 3.5), not an identity.  Returns (w_hard[B, L], dW[B, L],
    dc[S] or None) in float64."""
    st, _ = viterbi(w, c, n, k, nthreads)
    _, _, dW, dc = soft_codeword_vjp(w, c, n, k, T, g, want_dc, nthreads)
    return _d(c)[st], dW, dc


def block_tables(w_block, c, n, k, T, g_block=None):
    """One block: (log alpha[L, S], log beta[L, S], A[L, S] | None, B[L, S] | None)."""
    w = _d(w_block).reshape(-1)
    c = _d(c)
    L = w.shape[0]
    S = 1 << n
    al = np.empty((L, S), np.float64)
    be = np.empty((L, S), np.float64)
    A = Bt = None
    g = None
    if g_block is not None:
        g = _d(g_block).reshape(-1)
        A = np.empty((L, S), np.float64)
        Bt = np.empty((L, S), np.float64)
    rc = lib().oracle_block_tables(_ptr(w), L, _ptr(c), n, k, float(T), _ptr(g), _ptr(al),
                                   _ptr(be), _ptr(A), _ptr(Bt))
    _check(rc, "oracle_block_tables")
    return al, be, A, Bt

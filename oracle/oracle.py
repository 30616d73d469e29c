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
        L.oracle_soft_codeword_v.argtypes = [dp, i64, i64, dp, ci, ci, ci, cd, dp, dp, ci]
        L.oracle_soft_codeword_vjp_v.argtypes = [dp, i64, i64, dp, ci, ci, ci, cd, dp, dp, dp, dp,
                                                 dp, ci]
        L.oracle_viterbi_v.argtypes = [dp, i64, i64, dp, ci, ci, ci, ip, dp, ci]
        L.oracle_block_tables_v.argtypes = [dp, i64, dp, ci, ci, ci, cd, dp, dp, dp, dp, dp]
        L.oracle_maxmarginal_gap_v.argtypes = [dp, i64, i64, dp, ci, ci, ci, ip, dp, ci]
        for f in (L.oracle_soft_codeword, L.oracle_soft_codeword_vjp, L.oracle_viterbi,
                  L.oracle_block_tables, L.oracle_soft_codeword_v, L.oracle_soft_codeword_vjp_v,
                  L.oracle_viterbi_v, L.oracle_block_tables_v, L.oracle_maxmarginal_gap_v):
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


def _codebook(c, n, V):
    """Codebook as a flat float64 array of S*V values (state-major)."""
    c = _d(c).reshape(-1)
    if c.size != (1 << n) * V:
        raise ValueError(f"codebook must hold {1 << n} x {V} values, got {c.size}")
    return c


def soft_codeword(w, c, n, k, T, nthreads=None, V=1):
    """w[B, L] -> (w_soft[B, L] float64, logZ[B] float64).  With V > 1 each
    step emits V consecutive weights and c is [S, V] (or flat, state-major)."""
    w = _d(w)
    c = _codebook(c, n, V)
    B, L = w.shape
    ws = np.empty((B, L), np.float64)
    lz = np.empty((B,), np.float64)
    rc = lib().oracle_soft_codeword_v(_ptr(w), B, L, _ptr(c), n, k, V, float(T), _ptr(ws),
                                      _ptr(lz), nthreads or default_threads())
    _check(rc, "oracle_soft_codeword_v")
    return ws, lz


def soft_codeword_vjp(w, c, n, k, T, g, want_dc=True, nthreads=None, V=1):
    """Returns (w_soft, logZ, dW, dc) in float64; dc is summed over blocks
    (None when want_dc is False) and has the codebook's shape."""
    shape = np.shape(c)
    w = _d(w)
    c = _codebook(c, n, V)
    g = _d(g)
    B, L = w.shape
    assert g.shape == (B, L)
    ws = np.empty((B, L), np.float64)
    lz = np.empty((B,), np.float64)
    dW = np.empty((B, L), np.float64)
    dc = np.empty(c.size, np.float64) if want_dc else None
    rc = lib().oracle_soft_codeword_vjp_v(_ptr(w), B, L, _ptr(c), n, k, V, float(T), _ptr(g),
                                          _ptr(ws), _ptr(lz), _ptr(dW), _ptr(dc),
                                          nthreads or default_threads())
    _check(rc, "oracle_soft_codeword_vjp_v")
    return ws, lz, dW, (dc.reshape(shape) if want_dc else None)


def viterbi(w, c, n, k, nthreads=None, V=1):
    """w[B, L] -> (states[B, L // V] int32, cost[B] float64)."""
    w = _d(w)
    c = _codebook(c, n, V)
    B, L = w.shape
    st = np.empty((B, L // V), np.int32)
    cost = np.empty((B,), np.float64)
    rc = lib().oracle_viterbi_v(_ptr(w), B, L, _ptr(c), n, k, V, _ptr(st, ctypes.c_int32),
                                _ptr(cost), nthreads or default_threads())
    _check(rc, "oracle_viterbi_v")
    return st, cost


def maxmarginal_gap(w, c, n, k, states, nthreads=None, V=1):
    """Energy margin of the decoded codeword at every step (paper Sec. 3.2
    and the T -> 0 limit of Sec. 3.3): with M_t(s) the smallest distortion
    sum_tau ||w_tau - c(s_tau)||^2 of a legal path through s at step t,
    gap_t = (min over states emitting another codeword than c(states_t) of
    M_t(s) - M_t(states_t)) / 2, in the energy units of Eq. boltzmann.
    states[B, L // V] is a decoded path (``viterbi``).  float64 [B, L // V]."""
    w = _d(w)
    c = _codebook(c, n, V)
    B, L = w.shape
    st = np.ascontiguousarray(states, dtype=np.int32)
    assert st.shape == (B, L // V)
    gap = np.empty((B, L // V), np.float64)
    rc = lib().oracle_maxmarginal_gap_v(_ptr(w), B, L, _ptr(c), n, k, V,
                                        _ptr(st, ctypes.c_int32), _ptr(gap),
                                        nthreads or default_threads())
    _check(rc, "oracle_maxmarginal_gap_v")
    return gap


def crisp_positions(w, c, n, k, T, states, tol=2e-5, nthreads=None):
    """The T -> 0 check's excusal rule: a position must carry the decoded
    codeword (|w_soft_t - c(s*_t)| <= tol) when its max-marginal energy gap
    exceeds T ln(max |c_i - c_j| / tol), i.e. when the best competing
    codeword's Boltzmann weight, relative to the decoded one, times the
    largest codeword difference is below tol.  Returns (mask [B, L] of the
    positions held to the check, the gaps, the threshold)."""
    cf = np.asarray(c, np.float64).reshape(-1)
    spread = float(cf.max() - cf.min())
    thr = float(T) * np.log(spread / tol)
    gap = maxmarginal_gap(w, c, n, k, states, nthreads)
    return gap > thr, gap, thr


def ste(w, c, n, k, T, g, want_dc=True, nthreads=None, V=1):
    """BCJR-STE (paper Sec. 3.5 and Sec. "BCJR-STE variant"): the forward
    output is the hard codeword c(s_t) of the minimum-distortion path
    (Sec. 3.2) and the backward pass is the VJP of the temperature-T soft
    codeword (Sec. 3.5), not an identity.  Returns (w_hard[B, L], dW[B, L],
    dc[S] or None) in float64."""
    st, _ = viterbi(w, c, n, k, nthreads, V)
    _, _, dW, dc = soft_codeword_vjp(w, c, n, k, T, g, want_dc, nthreads, V)
    wh = _codebook(c, n, V).reshape(-1, V)[st].reshape(np.shape(w))
    return wh, dW, dc


def block_tables(w_block, c, n, k, T, g_block=None, V=1):
    """One block: (log alpha[N, S], log beta[N, S], A[N, S] | None, B[N, S] | None),
    N = L / V steps."""
    w = _d(w_block).reshape(-1)
    c = _codebook(c, n, V)
    L = w.shape[0]
    N = L // V
    S = 1 << n
    al = np.empty((N, S), np.float64)
    be = np.empty((N, S), np.float64)
    A = Bt = None
    g = None
    if g_block is not None:
        g = _d(g_block).reshape(-1)
        A = np.empty((N, S), np.float64)
        Bt = np.empty((N, S), np.float64)
    rc = lib().oracle_block_tables_v(_ptr(w), L, _ptr(c), n, k, V, float(T), _ptr(g), _ptr(al),
                                     _ptr(be), _ptr(A), _ptr(Bt))
    _check(rc, "oracle_block_tables_v")
    return al, be, A, Bt


# ---------------------------------------------------------------- computed codebook
_M64 = (1 << 64) - 1


def splitmix64(state: int):
    """SplitMix64 (Steele, Lea and Flood, 2014): returns (new state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & _M64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return state, z ^ (z >> 31)


def state_permutation(n: int, V: int, seed: int):
    """The V component permutations of the n-bit states: pi_a(s) with
    x = s * A1 + B, x ^= x >> h, x = x * A2, x ^= x >> h (mod 2^n,
    h = ceil(n / 2)), (A1 | 1, B, A2 | 1) consecutive SplitMix64 draws from
    seed.  Returns an int64 array [S, V]."""
    S = 1 << n
    mask = S - 1
    h = (n + 1) // 2
    st = seed & _M64
    s = np.arange(S, dtype=np.uint64)
    out = np.empty((S, V), np.int64)
    for a in range(V):
        st, a1 = splitmix64(st)
        st, b = splitmix64(st)
        st, a2 = splitmix64(st)
        a1 |= 1
        a2 |= 1
        with np.errstate(over="ignore"):
            x = (s * np.uint64(a1) + np.uint64(b)) & np.uint64(mask)
            x ^= x >> np.uint64(h)
            x = (x * np.uint64(a2)) & np.uint64(mask)
            x ^= x >> np.uint64(h)
        out[:, a] = x.astype(np.int64)
    return out


def gaussian_codebook(n: int, V: int, seed: int):
    """Computed Gaussian emission (paper Sec. 3.1): c_a(s) = Phi^{-1}((pi_a(s) +
    1/2) / S) under the incoherent permutation above.  float64 [S, V]
    (V = 1: [S])."""
    from scipy.special import ndtri
    S = 1 << n
    pi = state_permutation(n, V, seed)
    c = ndtri((pi.astype(np.float64) + 0.5) / S)
    return c[:, 0] if V == 1 else c


# ---------------------------------------------------------------- BlockLDLQ
def block_ldl(H, block):
    """H = M D M^T with M unit block-upper-triangular and D block-diagonal
    (blocks of `block`), from the Cholesky factor of H with its index order
    reversed (numpy, float64)."""
    H = np.asarray(H, np.float64)
    d = H.shape[0]
    R = np.linalg.cholesky(H[::-1, ::-1])[::-1, ::-1]     # H = R R^T, R upper triangular
    M = np.zeros_like(R)
    D = np.zeros_like(R)
    for k in range(0, d, block):
        Rkk = R[k:k + block, k:k + block]
        M[:, k:k + block] = R[:, k:k + block] @ np.linalg.inv(Rkk)
        D[k:k + block, k:k + block] = Rkk @ Rkk.T
    return M, D


def ldlq_viterbi(W, c, n, k, H, block, V=1, damp=0.01, targets_from=None):
    """BlockLDLQ rounding with the trellis quantiser (the PTQ reference of the
    paper's Eq. WPTQ for the Hessian-weighted loss, Eq. LHW): column blocks in
    order, block j rounded by Viterbi to the target
    t_j = w_j + sum_{i<j} (w_i - w_hat_i) M_ij.  H is damped by
    damp * mean(diag H).  Returns (W_hat, states[nb, rows, block // V],
    targets[nb, rows, block]) in float64.  With targets_from (a [rows, cols]
    W_hat) the targets are formed from that rounding instead of this one."""
    W = np.asarray(W, np.float64)
    rows, cols = W.shape
    Hd = np.asarray(H, np.float64)
    Hd = Hd + damp * np.mean(np.diag(Hd)) * np.eye(cols)
    M, _ = block_ldl(Hd, block)
    cb = _codebook(c, n, V).reshape(-1, V)
    nb = cols // block
    W_hat = np.zeros_like(W)
    states = np.zeros((nb, rows, block // V), np.int32)
    targets = np.zeros((nb, rows, block))
    for j in range(nb):
        sl = slice(j * block, (j + 1) * block)
        ref = W_hat if targets_from is None else np.asarray(targets_from, np.float64)
        t = W[:, sl] + (W[:, :j * block] - ref[:, :j * block]) @ M[:j * block, sl]
        targets[j] = t
        st, _ = viterbi(t, cb, n, k, V=V)
        states[j] = st
        W_hat[:, sl] = cb[st].reshape(rows, block)
    return W_hat, states, targets

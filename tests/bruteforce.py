"""Brute-force enumeration of every legal trellis path of a tiny block.

Independent of the oracle: it lists the S * K^(L-1) paths explicitly and
takes expectations under p_T(path) = exp(-E/T) / Z (paper Sec. 3.3,
Eq. boltzmann), with E = sum_t (w_t - c(s_t))^2 / 2 and
next(s, b) = ((s << k) | b) & (S - 1).  Used only as a pin for the oracle.
"""
import numpy as np


def paths(n, k, L):
    S, K = 1 << n, 1 << k
    st = np.arange(S, dtype=np.int64)[:, None]
    for _ in range(1, L):
        nxt = ((st[:, -1:] << k) & (S - 1))[:, None, :] + np.arange(K)[None, :, None]
        st = np.concatenate([np.repeat(st[:, None, :], K, axis=1), nxt], axis=2)
        st = st.reshape(-1, st.shape[-1])
    return st  # [S*K^(L-1), L]


def expectations(w, c, n, k, T, g=None, V=1):
    """One block.  Returns dict with logZ, w_soft[L], marg[N,S] and, with g,
    dW[L] = d<g,w_soft>/dw and dc = d<g,w_soft>/dc (shape of c), each
    computed as an exact path-level covariance.  With V > 1 every step emits
    V weights and c is [S, V]: the path's codeword is the concatenation of
    c(s_1), ..., c(s_N), N = L / V, and all sums run over the L components."""
    if V > 1:
        return _expectations_vec(w, c, n, k, T, g, V)
    w = np.asarray(w, np.float64)
    c = np.asarray(c, np.float64)
    L = w.shape[0]
    S = 1 << n
    P = paths(n, k, L)
    cP = c[P]                                   # c(s_t) per path
    E = 0.5 * ((w[None, :] - cP) ** 2).sum(1)
    a = -E / T
    m = a.max()
    wt = np.exp(a - m)
    Z = wt.sum()
    p = wt / Z
    out = {"logZ": m + np.log(Z)}
    out["w_soft"] = (p[:, None] * cP).sum(0)
    marg = np.zeros((L, S))
    for t in range(L):
        marg[t] = np.bincount(P[:, t], weights=p, minlength=S)
    out["marg"] = marg
    if g is not None:
        g = np.asarray(g, np.float64)
        F = (g[None, :] * cP).sum(1)
        EF = (p * F).sum()
        # d log p / d w_tau = -(w_tau - c(s_tau))/T + const  -> Cov(F, c(s_tau))/T
        out["dW"] = ((p * (F - EF))[:, None] * cP).sum(0) / T
        dc = np.zeros(S)
        for s in range(S):
            ind = (P == s)
            dF = (ind * g[None, :]).sum(1)                       # dF/dc_s
            dlog = (ind * (w[None, :] - c[s])).sum(1) / T        # d(-E/T)/dc_s
            dc[s] = (p * dF).sum() + (p * (F - EF) * (dlog - (p * dlog).sum())).sum()
        out["dc"] = dc
    return out


def _expectations_vec(w, c, n, k, T, g, V):
    w = np.asarray(w, np.float64)
    c = np.asarray(c, np.float64).reshape(1 << n, V)
    L = w.shape[0]
    N = L // V
    S = 1 << n
    P = paths(n, k, N)                          # [paths, N]
    cP = c[P].reshape(P.shape[0], L)            # emitted codeword per path
    E = 0.5 * ((w[None, :] - cP) ** 2).sum(1)
    a = -E / T
    m = a.max()
    wt = np.exp(a - m)
    Z = wt.sum()
    p = wt / Z
    out = {"logZ": m + np.log(Z), "w_soft": (p[:, None] * cP).sum(0)}
    marg = np.zeros((N, S))
    for t in range(N):
        marg[t] = np.bincount(P[:, t], weights=p, minlength=S)
    out["marg"] = marg
    if g is not None:
        g = np.asarray(g, np.float64)
        F = (g[None, :] * cP).sum(1)
        EF = (p * F).sum()
        out["dW"] = ((p * (F - EF))[:, None] * cP).sum(0) / T
        dc = np.zeros((S, V))
        for s in range(S):
            ind = np.repeat(P == s, V, axis=1)                  # [paths, L]
            for comp in range(V):
                sel = ind & (np.arange(L) % V == comp)[None, :]
                dF = (sel * g[None, :]).sum(1)
                dlog = (sel * (w[None, :] - c[s, comp])).sum(1) / T
                dc[s, comp] = (p * dF).sum() + (p * (F - EF) * (dlog - (p * dlog).sum())).sum()
        out["dc"] = dc
    return out


def viterbi_vec(w, c, n, k, V):
    """Vector-emission decode by enumeration: (best path [N], cost), the step
    distortion adding the V rounded squares in component order, steps
    summed left to right; ties as in viterbi()."""
    w = np.asarray(w, np.float64)
    c = np.asarray(c, np.float64).reshape(1 << n, V)
    N = w.shape[0] // V
    P = paths(n, k, N)
    cost = np.zeros(P.shape[0])
    for t in range(N):
        step = np.zeros(P.shape[0])
        for comp in range(V):
            d = w[t * V + comp] - c[P[:, t], comp]
            step = step + d * d
        cost = cost + step
    best = cost.min()
    cand = P[cost == best]
    order = np.lexsort(tuple(cand[:, t] for t in range(N)))
    return cand[order[0]], best


def viterbi(w, c, n, k):
    """All minimal-distortion paths; returns (best path chosen by the
    reverse-lexicographic rule: smallest s_L, then smallest s_{L-1}, ...,
    cost).  Distortions are summed left to right."""
    w = np.asarray(w, np.float64)
    c = np.asarray(c, np.float64)
    L = w.shape[0]
    P = paths(n, k, L)
    cost = np.zeros(P.shape[0])
    for t in range(L):
        d = w[t] - c[P[:, t]]
        cost = cost + d * d
    best = cost.min()
    cand = P[cost == best]
    order = np.lexsort(tuple(cand[:, t] for t in range(L)))  # last key (s_L) primary
    return cand[order[0]], best

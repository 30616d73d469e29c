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


def expectations(w, c, n, k, T, g=None):
    """One block.  Returns dict with logZ, w_soft[L], marg[L,S] and, with g,
    dW[L] = d<g,w_soft>/dw and dc[S] = d<g,w_soft>/dc, each computed as an
    exact path-level covariance."""
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

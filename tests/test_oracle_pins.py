"""Pins for the fp64 CPU oracle (runs without a GPU).

Each test ties the oracle to something other than itself: explicit path
enumeration, identities of the paper's equations, closed-form limits,
finite differences, or exact-arithmetic tie cases.
"""
import numpy as np
import pytest

import bruteforce as bf
from oracle import oracle as O

RNG = np.random.default_rng(20260510)

# (n, k, L): S = 2^n states, K = 2^k inputs per step, L steps.  Covers n >= 2k,
# n < 2k, n == k (fully connected) and k = 1, 3.
TINY = [(4, 2, 1), (4, 2, 2), (4, 2, 5), (4, 2, 6), (2, 1, 9), (3, 1, 10),
        (2, 2, 6), (3, 2, 6), (5, 2, 4), (4, 1, 8), (6, 3, 3), (3, 3, 4)]


def _case(n, k, L, seed):
    r = np.random.default_rng(seed)
    c = r.standard_normal(1 << n)
    w = r.standard_normal(L)
    g = r.standard_normal(L)
    return w, c, g


@pytest.mark.parametrize("n,k,L", TINY)
@pytest.mark.parametrize("T", [1.0, 0.25])
def test_forward_matches_enumeration(n, k, L, T):
    """Eq. soft-codeword and Z_T of Eq. boltzmann against all S*K^(L-1) paths."""
    w, c, _ = _case(n, k, L, 17 * n + 3 * k + L)
    ref = bf.expectations(w, c, n, k, T)
    ws, lz = O.soft_codeword(w[None], c, n, k, T)
    np.testing.assert_allclose(ws[0], ref["w_soft"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lz[0], ref["logZ"], rtol=1e-13, atol=1e-12)


@pytest.mark.parametrize("n,k,L", TINY)
def test_marginals_match_enumeration(n, k, L):
    """Eq. marginal: alpha_t(s) beta_t(s) / Z is the path marginal."""
    T = 0.6
    w, c, _ = _case(n, k, L, 5 * n + k + 11 * L)
    ref = bf.expectations(w, c, n, k, T)
    al, be, _, _ = O.block_tables(w, c, n, k, T)
    lz = O.soft_codeword(w[None], c, n, k, T)[1][0]
    p = np.exp(al + be - lz)
    np.testing.assert_allclose(p, ref["marg"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("n,k,L", TINY)
@pytest.mark.parametrize("T", [1.0, 0.3])
def test_vjp_matches_enumerated_covariances(n, k, L, T):
    """dW and dc against path-level covariances (derivative of Eq. boltzmann)."""
    w, c, g = _case(n, k, L, 101 * n + 7 * k + L)
    ref = bf.expectations(w, c, n, k, T, g)
    ws, lz, dW, dc = O.soft_codeword_vjp(w[None], c, n, k, T, g[None])
    scale = max(1.0, np.abs(ref["dW"]).max())
    np.testing.assert_allclose(dW[0], ref["dW"], rtol=0, atol=1e-11 * scale)
    scale = max(1.0, np.abs(ref["dc"]).max())
    np.testing.assert_allclose(dc, ref["dc"], rtol=0, atol=1e-11 * scale)
    np.testing.assert_allclose(ws[0], ref["w_soft"], atol=1e-12)


def test_partition_function_same_at_every_step():
    """Eq. marginal: Z = sum_s alpha_t(s) beta_t(s) for any t; marginals sum to 1."""
    n, k, L, T = 8, 2, 40, 0.2
    w, c, _ = _case(n, k, L, 3)
    al, be, _, _ = O.block_tables(w, c, n, k, T)
    lz = O.soft_codeword(w[None], c, n, k, T)[1][0]
    x = al + be
    m = x.max(1, keepdims=True)
    per_t = (m[:, 0] + np.log(np.exp(x - m).sum(1)))
    np.testing.assert_allclose(per_t, lz, rtol=1e-13)
    np.testing.assert_allclose(np.exp(x - lz).sum(1), 1.0, rtol=1e-12)


def _fd_logZ(w, c, n, k, T, h):
    L = w.shape[0]
    W = np.repeat(w[None], 2 * L, 0)
    for t in range(L):
        W[2 * t, t] += h
        W[2 * t + 1, t] -= h
    lz = O.soft_codeword(W, c, n, k, T)[1]
    return (lz[0::2] - lz[1::2]) / (2 * h)


@pytest.mark.parametrize("n,k", [(6, 2), (8, 2), (5, 1)])
def test_soft_codeword_is_gradient_of_logZ(n, k):
    """w_soft = w + T d logZ / dw  (Eq. boltzmann), by central differences of
    the forward-only log Z: pins w_soft independently of the beta sweep."""
    L, T = 12, 0.4
    w, c, _ = _case(n, k, L, 9 + n)
    ws = O.soft_codeword(w[None], c, n, k, T)[0][0]
    grad = _fd_logZ(w, c, n, k, T, 1e-5)
    np.testing.assert_allclose(ws, w + T * grad, rtol=0, atol=1e-8)


def _gdot(w, c, n, k, T, g):
    return (O.soft_codeword(w, c, n, k, T)[0] * g).sum()


@pytest.mark.parametrize("n,k,T", [(6, 2, 0.5), (8, 2, 0.2), (4, 1, 1.0)])
def test_vjp_matches_finite_differences(n, k, T):
    """dW and dc against central differences of <g, w_soft>."""
    B, L, h = 2, 10, 1e-5
    r = np.random.default_rng(n * 1000 + k)
    c = r.standard_normal(1 << n)
    w = r.standard_normal((B, L))
    g = r.standard_normal((B, L))
    _, _, dW, dc = O.soft_codeword_vjp(w, c, n, k, T, g)
    fd = np.zeros((B, L))
    for b in range(B):
        for t in range(L):
            wp = w.copy(); wp[b, t] += h
            wm = w.copy(); wm[b, t] -= h
            fd[b, t] = (_gdot(wp, c, n, k, T, g) - _gdot(wm, c, n, k, T, g)) / (2 * h)
    np.testing.assert_allclose(dW, fd, rtol=0, atol=2e-7 * max(1, np.abs(fd).max()))
    idx = r.choice(1 << n, size=12, replace=False)
    for s in idx:
        cp = c.copy(); cp[s] += h
        cm = c.copy(); cm[s] -= h
        f = (_gdot(w, cp, n, k, T, g) - _gdot(w, cm, n, k, T, g)) / (2 * h)
        assert abs(dc[s] - f) <= 2e-7 * max(1, abs(f)), (s, dc[s], f)


def test_jacobian_symmetric_and_psd():
    """J_{t,tau} = Cov(c(s_t), c(s_tau)) / T is symmetric positive semi-definite:
    g2 . VJP(g1) = g1 . VJP(g2) and g . VJP(g) >= 0."""
    n, k, L, T = 8, 2, 16, 0.15
    r = np.random.default_rng(4)
    c = r.standard_normal(1 << n)
    w = r.standard_normal((3, L))
    for _ in range(3):
        g1 = r.standard_normal((3, L))
        g2 = r.standard_normal((3, L))
        d1 = O.soft_codeword_vjp(w, c, n, k, T, g1, want_dc=False)[2]
        d2 = O.soft_codeword_vjp(w, c, n, k, T, g2, want_dc=False)[2]
        a, b = (g2 * d1).sum(), (g1 * d2).sum()
        assert abs(a - b) <= 1e-10 * max(1, abs(a))
        assert (g1 * d1).sum() >= -1e-12
    # full Jacobian of one block: symmetric, eigenvalues >= 0
    J = np.stack([O.soft_codeword_vjp(w[:1], c, n, k, T, np.eye(L)[i][None], want_dc=False)[2][0]
                  for i in range(L)])
    np.testing.assert_allclose(J, J.T, atol=1e-10 * np.abs(J).max())
    assert np.linalg.eigvalsh(0.5 * (J + J.T)).min() >= -1e-10 * np.abs(J).max()


def test_translation_invariance():
    """Shifting w and c together by a shifts w_soft by a, so
    sum(dW) + sum(dc) = sum(g) over the blocks of a call."""
    n, k, L, T = 8, 2, 20, 0.1
    r = np.random.default_rng(5)
    c = r.standard_normal(1 << n)
    w = r.standard_normal((4, L))
    g = r.standard_normal((4, L))
    _, _, dW, dc = O.soft_codeword_vjp(w, c, n, k, T, g)
    assert abs(dW.sum() + dc.sum() - g.sum()) <= 1e-9 * (np.abs(dW).sum() + np.abs(dc).sum())
    ws0 = O.soft_codeword(w, c, n, k, T)[0]
    ws1 = O.soft_codeword(w + 0.75, c + 0.75, n, k, T)[0]
    np.testing.assert_allclose(ws1, ws0 + 0.75, atol=1e-12)


def test_scaling():
    """(lam w, lam c, lam^2 T) gives lam * w_soft and the same log Z."""
    n, k, L, T, lam = 6, 2, 15, 0.3, 2.5
    r = np.random.default_rng(6)
    c = r.standard_normal(1 << n)
    w = r.standard_normal((3, L))
    ws0, lz0 = O.soft_codeword(w, c, n, k, T)
    ws1, lz1 = O.soft_codeword(lam * w, lam * c, n, k, lam * lam * T)
    np.testing.assert_allclose(ws1, lam * ws0, atol=1e-12)
    np.testing.assert_allclose(lz1, lz0, rtol=1e-12)


def test_high_temperature_limit():
    """T -> inf: every legal path equally likely; w_soft -> mean(c) and
    log Z + E_avg/T -> log(#paths) = log S + (L-1) k log 2."""
    n, k, L, T = 8, 2, 10, 1e9
    r = np.random.default_rng(7)
    c = r.standard_normal(1 << n)
    w = r.standard_normal(L)
    ws, lz = O.soft_codeword(w[None], c, n, k, T)
    np.testing.assert_allclose(ws[0], c.mean(), atol=1e-8)
    Eavg = 0.5 * ((w[:, None] - c[None, :]) ** 2).mean(1).sum()
    np.testing.assert_allclose(lz[0] + Eavg / T, n * np.log(2) + (L - 1) * k * np.log(2), atol=1e-8)


@pytest.mark.parametrize("n", [2, 3])
def test_fully_connected_trellis_is_independent_soft_quantizer(n):
    """n == k: every state reaches every state, so positions decouple:
    w_soft_t = sum_s c_s softmax_s(-(w_t - c_s)^2 / 2T) and the Jacobian is
    diagonal with J_tt = Var_t(c) / T."""
    k, L, T = n, 7, 0.4
    r = np.random.default_rng(8 + n)
    c = r.standard_normal(1 << n)
    w = r.standard_normal(L)
    g = r.standard_normal(L)
    ws, lz, dW, _ = O.soft_codeword_vjp(w[None], c, n, k, T, g[None])
    a = -(w[:, None] - c[None, :]) ** 2 / (2 * T)
    p = np.exp(a - a.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    mean = (p * c).sum(1)
    var = (p * c * c).sum(1) - mean ** 2
    np.testing.assert_allclose(ws[0], mean, atol=1e-13)
    np.testing.assert_allclose(dW[0], g * var / T, atol=1e-12)
    lz_ref = sum(np.log(np.exp(a[t] - a[t].max()).sum()) + a[t].max() for t in range(L))
    np.testing.assert_allclose(lz[0], lz_ref, rtol=1e-13)


def test_single_step_block():
    """L = 1: the marginal is a softmax over all S states."""
    n, k, T = 8, 2, 0.05
    r = np.random.default_rng(9)
    c = r.standard_normal(1 << n)
    w = r.standard_normal((5, 1))
    ws, lz = O.soft_codeword(w, c, n, k, T)
    a = -(w - c[None, :]) ** 2 / (2 * T)
    m = a.max(1, keepdims=True)
    p = np.exp(a - m)
    np.testing.assert_allclose(ws[:, 0], (p * c).sum(1) / p.sum(1), atol=1e-13)
    np.testing.assert_allclose(lz, m[:, 0] + np.log(p.sum(1)), rtol=1e-13)


@pytest.mark.parametrize("n,k,L", [(8, 2, 30), (6, 1, 25), (10, 2, 12)])
def test_low_temperature_marginals_concentrate_on_viterbi(n, k, L):
    """Sec. 3.3 identity 1: as T -> 0+ the Boltzmann distribution concentrates
    on the minimum-distortion path, so argmax_s p_t(s) is the Viterbi path."""
    T = 1e-9
    r = np.random.default_rng(n + 31 * L)
    c = r.standard_normal(1 << n)
    w = r.standard_normal(L)
    al, be, _, _ = O.block_tables(w, c, n, k, T)
    st, _ = O.viterbi(w[None], c, n, k)
    np.testing.assert_array_equal(np.argmax(al + be, 1), st[0])
    # at T = 1e-9 the log-domain values are ~1e9, so fp64 rounding alone
    # leaves ~1e-7 of normalisation error; check the value at T = 1e-6
    ws = O.soft_codeword(w[None], c, n, k, 1e-6)[0][0]
    np.testing.assert_allclose(ws, c[st[0]], atol=1e-8)


@pytest.mark.parametrize("n,k,L", [(4, 2, 6), (3, 1, 10), (5, 2, 5), (2, 2, 7), (6, 3, 3)])
def test_viterbi_matches_enumeration(n, k, L):
    r = np.random.default_rng(n * 7 + L)
    for _ in range(4):
        c = r.standard_normal(1 << n)
        w = r.standard_normal(L)
        st, cost = O.viterbi(w[None], c, n, k)
        p, best = bf.viterbi(w, c, n, k)
        np.testing.assert_array_equal(st[0], p)
        assert cost[0] == best


@pytest.mark.parametrize("n,k,L", [(4, 2, 6), (3, 1, 9), (4, 1, 8)])
def test_viterbi_tie_break_rule(n, k, L):
    """Exact ties (dyadic values; every sum is exact): the decode keeps the
    smallest final state, then the smallest predecessor at each step, i.e.
    the reverse-lexicographically smallest optimal path."""
    r = np.random.default_rng(n + k + L)
    for _ in range(6):
        c = r.integers(-3, 4, 1 << n) / 4.0      # many equal codewords
        w = r.integers(-6, 7, L) / 8.0
        st, cost = O.viterbi(w[None], c, n, k)
        p, best = bf.viterbi(w, c, n, k)
        np.testing.assert_array_equal(st[0], p)
        assert cost[0] == best


def test_monotone_in_own_weight():
    """d w_soft_t / d w_t = Var_p(c(s_t)) / T >= 0 (diagonal of the VJP)."""
    n, k, L, T = 8, 2, 12, 0.1
    r = np.random.default_rng(10)
    c = r.standard_normal(1 << n)
    w = r.standard_normal(L)
    al, be, _, _ = O.block_tables(w, c, n, k, T)
    lz = O.soft_codeword(w[None], c, n, k, T)[1][0]
    p = np.exp(al + be - lz)
    var = (p * c * c).sum(1) - ((p * c).sum(1)) ** 2
    for t in range(L):
        d = O.soft_codeword_vjp(w[None], c, n, k, T, np.eye(L)[t][None], want_dc=False)[2][0, t]
        assert d >= 0
        np.testing.assert_allclose(d, var[t] / T, rtol=1e-9, atol=1e-12)


def test_tangent_tables_are_conditional_expectations():
    """A_t(s) + B_t(s) = E[F | s_t = s] with F = sum_t g_t c(s_t), checked
    against the enumerated conditional expectation."""
    n, k, L, T = 4, 2, 5, 0.5
    w, c, g = _case(n, k, L, 12)
    _, _, A, Bt = O.block_tables(w, c, n, k, T, g)
    P = bf.paths(n, k, L)
    cP = c[P]
    a = -0.5 * ((w[None] - cP) ** 2).sum(1) / T
    p = np.exp(a - a.max()); p /= p.sum()
    F = (g[None] * cP).sum(1)
    for t in range(L):
        for s in range(1 << n):
            sel = P[:, t] == s
            ref = (p[sel] * F[sel]).sum() / p[sel].sum()
            assert abs(A[t, s] + Bt[t, s] - ref) <= 1e-11 * max(1, abs(ref))


def test_oracle_rejects_bad_arguments():
    c = np.zeros(16)
    w = np.zeros((1, 4))
    with pytest.raises(RuntimeError):
        O.soft_codeword(w, c, 4, 5, 1.0)     # k > n
    with pytest.raises(RuntimeError):
        O.soft_codeword(w, c, 4, 2, 0.0)     # T <= 0
    with pytest.raises(RuntimeError):
        O.soft_codeword(w, c, 4, 2, float("nan"))


@pytest.mark.parametrize("n,k,L", [(4, 2, 5), (3, 1, 8), (5, 2, 4), (6, 3, 3)])
@pytest.mark.parametrize("T", [0.7, 0.1])
def test_ste_matches_enumeration(n, k, L, T):
    """BCJR-STE: forward = codeword of the enumerated minimum-distortion path
    (independent of T); backward = enumerated path covariances at T."""
    for seed in range(3):
        w, c, g = _case(n, k, L, 4242 + 31 * seed + n)
        wh, dW, dc = O.ste(w[None], c, n, k, T, g[None])
        p, _ = bf.viterbi(w, c, n, k)
        np.testing.assert_array_equal(wh[0], c[p])
        ref = bf.expectations(w, c, n, k, T, g)
        np.testing.assert_allclose(dW[0], ref["dW"], rtol=0, atol=1e-10 * max(1, abs(ref["dW"]).max()))
        np.testing.assert_allclose(dc, ref["dc"], rtol=0, atol=1e-10 * max(1, abs(ref["dc"]).max()))


def test_ste_gradient_couples_neighbours():
    """The STE backward is the trellis-coupled gradient, not the identity:
    a unit upstream gradient at step t moves dW at other steps, and its own
    entry is Var(c(s_t))/T, not 1."""
    n, k, L, T = 4, 2, 8, 0.3       # 16 * 4^7 enumerated paths
    w, c, _ = _case(n, k, L, 77)
    t = 4
    g = np.zeros(L); g[t] = 1.0
    _, dW, _ = O.ste(w[None], c, n, k, T, g[None], want_dc=False)
    ref = bf.expectations(w, c, n, k, T)
    var_t = (ref["marg"][t] * c * c).sum() - ref["w_soft"][t] ** 2
    assert abs(dW[0, t] - var_t / T) <= 1e-10 * max(1.0, var_t / T)
    assert abs(dW[0, t - 1]) > 1e-6 and abs(dW[0, t + 1]) > 1e-6


# ---------------------------------------------------------------- V = 2
# Vector emission (Sec. 3.1 with V = 2; the kV = 4, 16-predecessor trellis of
# Sec. 4.1 is (n, k) = (16, 4)).  (n, k, L weights): K = 16 cases keep the
# enumeration small (S * 16^(N-1) paths).
VEC = [(8, 4, 4), (6, 4, 6), (4, 4, 6), (4, 2, 8), (3, 1, 10), (5, 2, 6)]


def _vcase(n, L, seed, V=2):
    r = np.random.default_rng(seed)
    return r.standard_normal(L), r.standard_normal((1 << n, V)), r.standard_normal(L)


@pytest.mark.parametrize("n,k,L", VEC)
@pytest.mark.parametrize("T", [1.0, 0.2])
def test_vector_emission_matches_enumeration(n, k, L, T):
    for seed in range(2):
        w, c, g = _vcase(n, L, 900 + 17 * seed + n * k)
        ws, lz, dW, dc = O.soft_codeword_vjp(w[None], c, n, k, T, g[None], V=2)
        ref = bf.expectations(w, c, n, k, T, g, V=2)
        tol = lambda a: 1e-10 * max(1.0, np.abs(a).max())
        assert abs(lz[0] - ref["logZ"]) <= 1e-10 * max(1.0, abs(ref["logZ"]))
        np.testing.assert_allclose(ws[0], ref["w_soft"], rtol=0, atol=1e-11)
        np.testing.assert_allclose(dW[0], ref["dW"], rtol=0, atol=tol(ref["dW"]))
        np.testing.assert_allclose(dc, ref["dc"], rtol=0, atol=tol(ref["dc"]))
        al, be, _, _ = O.block_tables(w, c, n, k, T, V=2)
        marg = np.exp(al + be - lz[0])
        np.testing.assert_allclose(marg, ref["marg"], rtol=0, atol=1e-11)


@pytest.mark.parametrize("n,k,T", [(8, 4, 0.3), (6, 2, 0.5)])
def test_vector_vjp_matches_finite_differences(n, k, T):
    B, L, h = 2, 12, 1e-5
    r = np.random.default_rng(31 * n + k)
    c = r.standard_normal((1 << n, 2))
    w = r.standard_normal((B, L))
    g = r.standard_normal((B, L))
    _, _, dW, dc = O.soft_codeword_vjp(w, c, n, k, T, g, V=2)

    def gdot(w_, c_):
        return (O.soft_codeword(w_, c_, n, k, T, V=2)[0] * g).sum()

    for b in range(B):
        for t in range(L):
            wp = w.copy(); wp[b, t] += h
            wm = w.copy(); wm[b, t] -= h
            fd = (gdot(wp, c) - gdot(wm, c)) / (2 * h)
            assert abs(dW[b, t] - fd) <= 2e-7 * max(1, abs(fd)), (b, t, dW[b, t], fd)
    for s in r.choice(1 << n, size=8, replace=False):
        for comp in range(2):
            cp = c.copy(); cp[s, comp] += h
            cm = c.copy(); cm[s, comp] -= h
            fd = (gdot(w, cp) - gdot(w, cm)) / (2 * h)
            assert abs(dc[s, comp] - fd) <= 2e-7 * max(1, abs(fd)), (s, comp, dc[s, comp], fd)


def test_vector_emission_with_constant_component_reduces_to_scalar():
    """c(s) = (c0(s), const): the second weights of every step see the same
    energy on every path, so the distribution is the scalar trellis on the
    first weights; the second components' soft codeword is the constant and
    their dW is 0."""
    n, k, L, T = 8, 4, 16, 0.25
    r = np.random.default_rng(5)
    c0 = r.standard_normal(1 << n)
    c = np.stack([c0, np.full(1 << n, 0.375)], axis=1)
    w = r.standard_normal((3, L))
    g = r.standard_normal((3, L))
    ws, lz, dW, dc = O.soft_codeword_vjp(w, c, n, k, T, g, V=2)
    ws1, lz1, dW1, dc1 = O.soft_codeword_vjp(w[:, 0::2], c0, n, k, T, g[:, 0::2])
    np.testing.assert_allclose(ws[:, 0::2], ws1, rtol=0, atol=1e-12)
    np.testing.assert_allclose(ws[:, 1::2], 0.375, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dW[:, 0::2], dW1, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dW[:, 1::2], 0.0, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dc[:, 0], dc1, rtol=0, atol=1e-11)
    # logZ differs by the constant energy of the second weights
    shift = -(((w[:, 1::2] - 0.375) ** 2).sum(1)) / (2 * T)
    np.testing.assert_allclose(lz, lz1 + shift, rtol=0, atol=1e-10)
    # dc of the constant component: sum over steps of g_t,1 + (w_t,1 - c)(...)
    # only its total over states is fixed: sum_s p_t(s) = 1 at every step
    np.testing.assert_allclose(dc[:, 1].sum(), g[:, 1::2].sum(), rtol=0, atol=1e-9)


@pytest.mark.parametrize("n,k,L", [(8, 4, 6), (4, 4, 8), (5, 2, 10), (3, 1, 12)])
def test_vector_viterbi_matches_enumeration(n, k, L):
    r = np.random.default_rng(n * 13 + L)
    for _ in range(3):
        w, c, _ = _vcase(n, L, int(r.integers(1 << 30)))
        st, cost = O.viterbi(w[None], c, n, k, V=2)
        p, best = bf.viterbi_vec(w, c, n, k, 2)
        np.testing.assert_array_equal(st[0], p)
        assert cost[0] == best


@pytest.mark.parametrize("n,k,L", [(8, 4, 6), (4, 2, 8)])
def test_vector_viterbi_tie_break_rule(n, k, L):
    """Dyadic values (every sum exact): many exact ties, resolved to the
    reverse-lexicographically smallest optimal path."""
    r = np.random.default_rng(n + k + L + 1)
    for _ in range(4):
        c = r.integers(-3, 4, (1 << n, 2)) / 4.0
        w = r.integers(-6, 7, L) / 8.0
        st, cost = O.viterbi(w[None], c, n, k, V=2)
        p, best = bf.viterbi_vec(w, c, n, k, 2)
        np.testing.assert_array_equal(st[0], p)
        assert cost[0] == best


def test_vector_ste_composition():
    n, k, L, T = 6, 4, 6, 0.4
    w, c, g = _vcase(n, L, 4711)
    wh, dW, dc = O.ste(w[None], c, n, k, T, g[None], V=2)
    p, _ = bf.viterbi_vec(w, c, n, k, 2)
    np.testing.assert_array_equal(wh[0], c[p].reshape(-1))
    ref = bf.expectations(w, c, n, k, T, g, V=2)
    np.testing.assert_allclose(dW[0], ref["dW"], rtol=0, atol=1e-10 * max(1, abs(ref["dW"]).max()))



# ---------------------------------------------------------------- computed codebook
def test_splitmix64_reference_outputs():
    """The first outputs of SplitMix64 started from state 0, as printed by its
    reference C implementation (Vigna)."""
    st, out = 0, []
    for _ in range(3):
        st, z = O.splitmix64(st)
        out.append(z)
    assert out == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


@pytest.mark.parametrize("n,V", [(1, 1), (4, 2), (8, 1), (12, 2), (16, 2), (17, 3)])
def test_state_permutation_is_a_bijection(n, V):
    pi = O.state_permutation(n, V, 20260510)
    for a in range(V):
        assert np.array_equal(np.sort(pi[:, a]), np.arange(1 << n))
    if n >= 8:  # incoherent: neighbouring states land far apart
        d = np.abs(np.diff(pi[:, 0]))
        assert np.median(d) > (1 << n) / 16


@pytest.mark.parametrize("n,V", [(4, 1), (10, 2), (16, 2)])
def test_gaussian_codebook_is_the_normal_quantiles(n, V):
    """Sorted, each component is the S Gaussian quantiles: Phi(c_(i)) = (i + 1/2)/S
    with Phi from the error function, and the quantiles are symmetric."""
    import math
    c = O.gaussian_codebook(n, V, 7).reshape(1 << n, V)
    S = 1 << n
    for a in range(V):
        q = np.sort(c[:, a])
        phi = np.array([0.5 * math.erfc(-x / math.sqrt(2.0)) for x in q])
        np.testing.assert_allclose(phi, (np.arange(S) + 0.5) / S, rtol=1e-12, atol=0)
        np.testing.assert_allclose(q, -q[::-1], rtol=0, atol=1e-12)
    assert abs(c.mean()) < 1e-12
    if n >= 10:
        assert abs(c.var() - 1) < 0.01



# ---------------------------------------------------------------- BlockLDLQ
def _hessian(d, seed, n_x=None):
    r = np.random.default_rng(seed)
    n_x = n_x or 4 * d
    X = r.standard_normal((n_x, d)) @ (np.eye(d) + 0.7 * r.standard_normal((d, d)) / np.sqrt(d))
    return X.T @ X / n_x


def test_block_ldl_factorisation():
    H = _hessian(48, 1)
    M, D = O.block_ldl(H, 16)
    np.testing.assert_allclose(M @ D @ M.T, H, rtol=0, atol=1e-12 * np.abs(H).max())
    assert np.abs(np.tril(M, -1)).max() == 0.0
    for k in range(0, 48, 16):
        np.testing.assert_allclose(M[k:k + 16, k:k + 16], np.eye(16), rtol=0, atol=1e-12)
    for k in range(0, 48, 16):
        D[k:k + 16, k:k + 16] = 0
    assert np.abs(D).max() == 0.0


def test_ldlq_loss_identity():
    """e H e^T = sum_k (e M)_k D_k (e M)_k^T for any error e: the quantity the
    block-by-block rounding controls."""
    H = _hessian(32, 2)
    M, D = O.block_ldl(H, 8)
    e = np.random.default_rng(3).standard_normal((5, 32))
    lhs = np.einsum("ri,ij,rj->r", e, H, e)
    eM = e @ M
    rhs = sum(np.einsum("ri,ij,rj->r", eM[:, k:k + 8], D[k:k + 8, k:k + 8], eM[:, k:k + 8])
              for k in range(0, 32, 8))
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12)


def test_ldlq_reduces_to_plain_viterbi():
    """H = I (no coupling between blocks) and a single block both give the
    plain per-block Viterbi codeword."""
    n, k = 6, 2
    r = np.random.default_rng(4)
    c = r.standard_normal(1 << n)
    W = r.standard_normal((3, 24))
    plain, _ = O.viterbi(W.reshape(-1, 8), c, n, k)
    Wh, _, _ = O.ldlq_viterbi(W, c, n, k, np.eye(24), 8, damp=0.0)
    np.testing.assert_array_equal(Wh.reshape(-1, 8), c[plain])
    H = _hessian(24, 5)
    st1, _ = O.viterbi(W, c, n, k)
    Wh1, _, _ = O.ldlq_viterbi(W, c, n, k, H, 24)
    np.testing.assert_array_equal(Wh1, c[st1])


def test_ldlq_lowers_the_hessian_weighted_loss():
    n, k, block = 6, 2, 8
    r = np.random.default_rng(6)
    c = r.standard_normal(1 << n)
    W = r.standard_normal((16, 48))
    H = _hessian(48, 7)
    Wh, _, _ = O.ldlq_viterbi(W, c, n, k, H, block, damp=0.0)
    st, _ = O.viterbi(W.reshape(-1, block), c, n, k)
    plain = c[st].reshape(W.shape)
    loss = lambda X: np.einsum("ri,ij,rj->", W - X, H, W - X)
    assert loss(Wh) < 0.9 * loss(plain)


# ---------------------------------------------------------------- T -> 0 check
def _path_costs(w, c, n, k, V=1):
    """Every legal path and its distortion, summed step by step."""
    c = np.asarray(c, np.float64).reshape(1 << n, V)
    N = len(w) // V
    P = bf.paths(n, k, N)
    cost = np.zeros(P.shape[0])
    for t in range(N):
        step = np.zeros(P.shape[0])
        for comp in range(V):
            d = w[t * V + comp] - c[P[:, t], comp]
            step = step + d * d
        cost = cost + step
    return P, cost, c


@pytest.mark.parametrize("n,k,L,V", [(4, 2, 6, 1), (3, 1, 9, 1), (5, 2, 5, 1), (6, 3, 3, 1),
                                     (4, 2, 8, 2), (8, 4, 6, 2)])
def test_maxmarginal_gap_matches_enumeration(n, k, L, V):
    """gap_t = (min over paths whose step-t codeword differs from the decoded
    one of their distortion - the optimal distortion) / 2, by listing every
    path."""
    r = np.random.default_rng(100 * n + 10 * k + L + V)
    for _ in range(3):
        c = r.standard_normal((1 << n) * V)
        w = r.standard_normal(L)
        st, _ = O.viterbi(w[None], c, n, k, V=V)
        gap = O.maxmarginal_gap(w[None], c, n, k, st, V=V)[0]
        P, cost, cv = _path_costs(w, c, n, k, V)
        best = cost.min()
        for t in range(L // V):
            other = np.any(cv[P[:, t]] != cv[st[0, t]][None, :], axis=1)
            ref = 0.5 * (cost[other].min() - best)
            np.testing.assert_allclose(gap[t], ref, rtol=1e-12, atol=1e-12)
            assert gap[t] >= 0


def test_maxmarginal_gap_ignores_states_with_the_same_codeword():
    """Dyadic codebook with repeated values: a competing path that only
    changes the state, not the emitted codeword, is not a competitor; with
    every codeword equal the gap is infinite."""
    n, k, L = 4, 2, 7
    r = np.random.default_rng(77)
    for _ in range(4):
        c = r.integers(-2, 3, 1 << n) / 4.0
        w = r.integers(-6, 7, L) / 8.0
        st, _ = O.viterbi(w[None], c, n, k)
        gap = O.maxmarginal_gap(w[None], c, n, k, st)[0]
        P, cost, cv = _path_costs(w, c, n, k)
        for t in range(L):
            other = cv[P[:, t], 0] != c[st[0, t]]
            assert gap[t] == 0.5 * (cost[other].min() - cost.min())
    const = np.full(1 << n, 0.5)
    st, _ = O.viterbi(w[None], const, n, k)
    assert np.all(np.isinf(O.maxmarginal_gap(w[None], const, n, k, st)))


def test_maxmarginal_gap_bounds_the_soft_codeword_deviation():
    """At low T the soft codeword leaves the decoded codeword by at most
    (number of paths) x max|c_i - c_j| x exp(-gap / T) (every competing path
    has energy at least gap above the best one), and by at least
    |c_alt - c*| exp(-gap / T) p* for the best competitor, so the rule that
    holds a position to the check when gap > T ln(max|dc| / tol) is tied to
    the Boltzmann weights of Eq. boltzmann."""
    n, k, L, T = 4, 2, 6, 0.02
    r = np.random.default_rng(5)
    c = r.standard_normal(1 << n)
    w = r.standard_normal(L)
    st, _ = O.viterbi(w[None], c, n, k)
    gap = O.maxmarginal_gap(w[None], c, n, k, st)[0]
    ws = O.soft_codeword(w[None], c, n, k, T)[0][0]
    npaths = (1 << n) * (1 << k) ** (L - 1)
    spread = c.max() - c.min()
    dev = np.abs(ws - c[st[0]])
    assert np.all(dev <= npaths * spread * np.exp(-gap / T) + 1e-15)
    mask, _, thr = O.crisp_positions(w[None], c, n, k, T, st, tol=1e-3)
    np.testing.assert_allclose(thr, T * np.log(spread / 1e-3))
    assert np.array_equal(mask[0], gap > thr)

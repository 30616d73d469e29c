"""The minimum-distortion decode's tie rule on the GPU (paper Sec. 3.2; the
paper leaves ties open, the reading taken is: among equal path metrics the
predecessor with the smallest state index, then the smallest final state).

Inputs are dyadic (codewords in {-3..3}/4, weights in {-6..6}/8), so every
fp64 distortion and every metric sum is exact on both sides and exact ties
are everywhere: the states must equal the oracle's bit for bit (the
oracle's rule is pinned against path enumeration on tiny shapes), and
w_hard must be codebook[states].
"""
import sys

import numpy as np
import pytest

import paper_2605_10655_amd as P
from oracle import oracle as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P.load_library()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def host(t):
    return t.detach().cpu().numpy()


def dyadic(seed, B, L, S, V=1):
    r = np.random.default_rng(seed)
    c = (r.integers(-3, 4, (S, V) if V > 1 else S) / 4.0).astype(np.float32)
    w = (r.integers(-6, 7, (B, L)) / 8.0).astype(np.float32)
    return w, c


@pytest.mark.parametrize("n,k,B,L", [
    (2, 1, 9, 14), (6, 1, 7, 12), (10, 1, 5, 11), (14, 1, 3, 9),
    (4, 2, 9, 13), (8, 2, 7, 12), (12, 2, 5, 10), (13, 2, 3, 9), (16, 2, 3, 9),
    (6, 3, 6, 10), (9, 3, 4, 8), (14, 3, 2, 7),
])
def test_scalar_viterbi_tie_rule(n, k, B, L):
    w, c = dyadic(17 * n + k, B, L, 1 << n)
    _say(f"[ties] scalar n={n} k={k} B={B} L={L}")
    st, wh = P.viterbi_decode(dev(w), dev(c), n, k)
    torch.cuda.synchronize()
    st, wh = host(st), host(wh)
    rst, cost = O.viterbi(w, c, n, k)
    np.testing.assert_array_equal(st, rst)
    np.testing.assert_array_equal(wh, c[st])
    # the inputs really tie: some step has several states of the best metric
    m = O.maxmarginal_gap(w, c, n, k, rst)
    assert np.any(m == 0.0)


@pytest.mark.parametrize("n,B,L", [(8, 6, 12), (12, 4, 10), (16, 2, 8)])
def test_vector_viterbi_tie_rule(n, B, L):
    w, c = dyadic(31 * n, B, L, 1 << n, V=2)
    _say(f"[ties] vector n={n} V=2 B={B} L={L}")
    st, wh = P.bcjr_vec_viterbi_decode(dev(w), dev(c), n, 4, 2)
    torch.cuda.synchronize()
    st, wh = host(st), host(wh)
    rst, _ = O.viterbi(w, c, n, 4, V=2)
    np.testing.assert_array_equal(st, rst)
    np.testing.assert_array_equal(wh, c[st].reshape(B, L))
    assert np.any(O.maxmarginal_gap(w, c, n, 4, rst, V=2) == 0.0)

"""GPU parity of the fp64 generic family (bcjr_generic_kernels.h): the
trellis shapes outside the super-group kernels -- fewer state bits than two
shift digits (n < 2k, down to the fully connected n = k), shifts of 4 or more
bits with scalar emission, and 15-16 state bits at k = 1 and k = 3 -- against
the fp64 oracle on the same seeded inputs.

Tolerances as everywhere: w_soft |err| <= 2e-5, logZ 1e-4 relative, dW and
dCodebook 1e-4 of max(|ref_i|, rms(ref)); Viterbi states bit-exact and
w_hard == codebook[states], including exact ties (dyadic inputs).
"""
import sys

import numpy as np
import pytest

import paper_2605_10655_amd as P
from paper_2605_10655_amd import workloads as WL
from oracle import oracle as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL_WS, TOL_LOGZ, TOL_GRAD = 2e-5, 1e-4, 1e-4

# (n, k, B, L): n = k, n < 2k, k >= 4, k = 1 and k = 3 at 15-16 state bits
SHAPES = [
    (1, 1, 5, 9), (2, 2, 4, 7), (3, 2, 6, 11), (4, 3, 5, 8), (5, 3, 3, 10), (4, 4, 3, 6),
    (6, 4, 4, 9), (8, 4, 3, 12), (9, 5, 2, 7), (12, 6, 2, 6), (10, 10, 2, 5), (8, 8, 3, 6),
    (15, 1, 2, 7), (16, 1, 2, 6), (15, 3, 2, 6), (16, 3, 2, 5), (16, 4, 2, 4),
]


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


def grad_err(gpu, ref):
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt(np.mean(ref * ref))
    scale = np.maximum(np.abs(ref), rms)
    return float((np.abs(gpu.astype(np.float64) - ref) / np.where(scale > 0, scale, 1.0)).max())


def check(w, c, n, k, T, g, what, workspace=None):
    out = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), n, k, T, dev(g), workspace=workspace)
    torch.cuda.synchronize()
    ws, lz, dW, dc = (host(t) for t in out)
    rws, rlz, rdW, rdc = O.soft_codeword_vjp(w, c, n, k, float(np.float32(T)), g)
    e = (float(np.abs(ws - rws).max()), float((np.abs(lz - rlz) / np.abs(rlz)).max()),
         grad_err(dW, rdW), grad_err(dc, rdc))
    _say(f"[generic] {what}: w_soft {e[0]:.2e} logZ {e[1]:.2e} dW {e[2]:.2e} dc {e[3]:.2e}")
    assert e[0] <= TOL_WS and e[1] <= TOL_LOGZ and e[2] <= TOL_GRAD and e[3] <= TOL_GRAD
    return ws, lz, dW, dc


@pytest.mark.parametrize("n,k,B,L", SHAPES)
@pytest.mark.parametrize("T", [0.3, 0.003])
def test_generic_shapes_match_oracle(n, k, B, L, T):
    w, c, g = WL.random_case(7000 + 37 * n + k, B, L, n)
    ws, _, _, _ = check(w, c, n, k, T, g, f"n={n} k={k} B={B} L={L} T={T}")
    # the soft codeword alone and the separate VJP give the same numbers
    sws, _ = P.bcjr_soft_codeword(dev(w), dev(c), n, k, T)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(sws), ws)
    st, wh = P.viterbi_decode(dev(w), dev(c), n, k)
    torch.cuda.synchronize()
    rst, _ = O.viterbi(w, c, n, k)
    np.testing.assert_array_equal(host(st), rst)
    np.testing.assert_array_equal(host(wh), c[rst])


@pytest.mark.parametrize("n,k,B,L", [(3, 2, 7, 12), (5, 3, 5, 10), (4, 4, 4, 9), (8, 4, 3, 10),
                                     (16, 1, 2, 8), (15, 3, 2, 7)])
def test_generic_viterbi_tie_rule(n, k, B, L):
    r = np.random.default_rng(55 * n + k)
    c = (r.integers(-3, 4, 1 << n) / 4.0).astype(np.float32)
    w = (r.integers(-6, 7, (B, L)) / 8.0).astype(np.float32)
    st, wh = P.viterbi_decode(dev(w), dev(c), n, k)
    torch.cuda.synchronize()
    rst, _ = O.viterbi(w, c, n, k)
    np.testing.assert_array_equal(host(st), rst)
    np.testing.assert_array_equal(host(wh), c[rst])
    assert np.any(O.maxmarginal_gap(w, c, n, k, rst) == 0.0)


def test_generic_persistent_loop_and_ste():
    """A workspace of one slot makes one workgroup walk every block: same
    bits as the full-size run; bcjr_ste_vjp gives the fused call's dW and
    dCodebook (the generic family has no centring reference to use)."""
    n, k, B, L, T = 6, 4, 9, 14, 0.05
    w, c, g = WL.random_case(8080, B, L, n)
    full = check(w, c, n, k, T, g, "one-slot reference")
    big = P.bcjr_workspace_bytes(B, L, n, k, P.OP_FWD_VJP)
    small = torch.empty(big // B, dtype=torch.uint8, device="cuda:0")
    one = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), n, k, T, dev(g), workspace=small)
    torch.cuda.synchronize()
    for a, b in zip(full[:3], one[:3]):
        np.testing.assert_array_equal(a, host(b))
    d = np.abs(full[3].astype(np.float64) - host(one[3]))
    assert d.max() <= 4 * 2.0 ** -24 * np.abs(full[3]).max()
    _, wh = P.viterbi_decode(dev(w), dev(c), n, k)
    sdW, sdc = P.bcjr_ste_vjp(dev(w), dev(c), n, k, T, wh, dev(g))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(sdW), full[2])
    np.testing.assert_array_equal(host(sdc), full[3])


def test_generic_empty_batch_and_one_step():
    n, k = 5, 3
    c = dev(np.linspace(-1, 1, 1 << n).astype(np.float32))
    dc = torch.full((1 << n,), 3.0, device="cuda:0")
    e = torch.empty((0, 4), dtype=torch.float32, device="cuda:0")
    P.bcjr_soft_codeword_vjp(e, c, n, k, 1.0, e, want_dW=False, dCodebook=dc,
                             workspace=torch.empty(256, dtype=torch.uint8, device="cuda:0"))
    torch.cuda.synchronize()
    assert float(dc.abs().max()) == 0.0
    w, cc, g = WL.random_case(99, 4, 1, n)     # L = 1: softmax over all states
    check(w, cc, n, k, 0.7, g, "L=1")

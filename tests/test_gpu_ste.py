"""GPU parity of the autograd layer and the BCJR-STE variant against the
fp64 oracle.

BCJR-STE: forward = hard Viterbi codeword (bit-exact against the oracle's
decode), backward = VJP of the soft codeword at T (same tolerance as the soft
VJP: |gpu - ref| <= 1e-4 max(|ref_i|, rms(ref))).  bcjr_ste_vjp fed with the
forward's codewords must reproduce bcjr_soft_codeword_vjp bit for bit on both
sides of the precision switch.
"""
import sys

import numpy as np
import pytest

import paper_2605_10655_amd as P
from paper_2605_10655_amd import workloads as WL
from oracle import oracle as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL_WS = 2e-5
TOL_GRAD = 1e-4


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P.load_library()
    yield


def dev(a, grad=False):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0").requires_grad_(grad)


def host(t):
    return None if t is None else t.detach().cpu().numpy()


def check_grad(gpu, ref, what=""):
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt(np.mean(ref * ref))
    scale = np.maximum(np.abs(ref), rms)
    err = (np.abs(gpu.astype(np.float64) - ref) / np.where(scale > 0, scale, 1.0)).max()
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite gradient"
    assert err <= TOL_GRAD, f"{what}: gradient err {err:.3e} (rms {rms:.3e})"
    return err


def autograd_step(w, c, n, k, T, g, hard, block=None):
    """Forward through BcjrQuant (or bcjr_quant with a block size), then
    backward with upstream g: (out, dW, dc) on the host."""
    from paper_2605_10655_amd.autograd import BcjrQuant, bcjr_quant
    wt, ct = dev(w, True), dev(c, True)
    if block is None:
        out = BcjrQuant.apply(wt, ct, n, k, T, hard)
    else:
        out = bcjr_quant(wt, ct, n, k, T, block=block, hard=hard)
    out.backward(dev(g))
    torch.cuda.synchronize()
    return host(out), host(wt.grad), host(ct.grad)


CASES = [(4, 2, 9, 16), (8, 2, 5, 40), (12, 2, 3, 30), (16, 2, 2, 12), (6, 1, 7, 21),
         (8, 3, 3, 9)]


@pytest.mark.parametrize("n,k,B,L", CASES)
@pytest.mark.parametrize("T", [0.3, 0.05, 0.003])
def test_ste_autograd_matches_oracle(n, k, B, L, T):
    w, c, g = WL.random_case(7000 + 100 * n + 10 * k + B, B, L, n)
    _say(f"[ste] n={n} k={k} B={B} L={L} T={T}")
    out, dW, dc = autograd_step(w, c, n, k, T, g, hard=True)
    rwh, rdW, rdc = O.ste(w, c, n, k, float(np.float32(T)), g)
    np.testing.assert_array_equal(out, rwh.astype(np.float32))
    e = (check_grad(dW, rdW, "ste dW"), check_grad(dc, rdc, "ste dc"))
    _say(f"[ste] errors {['%.2e' % x for x in e]}")


@pytest.mark.parametrize("n,k,B,L", CASES[:4])
@pytest.mark.parametrize("T", [0.3, 0.003])
def test_soft_autograd_matches_oracle(n, k, B, L, T):
    w, c, g = WL.random_case(8000 + 100 * n + 10 * k + B, B, L, n)
    _say(f"[soft autograd] n={n} k={k} B={B} L={L} T={T}")
    out, dW, dc = autograd_step(w, c, n, k, T, g, hard=False)
    rws, _, rdW, rdc = O.soft_codeword_vjp(w, c, n, k, float(np.float32(T)), g)
    assert np.abs(out.astype(np.float64) - rws).max() <= TOL_WS
    check_grad(dW, rdW, "soft dW")
    check_grad(dc, rdc, "soft dc")


@pytest.mark.parametrize("T", [0.2, 0.01])
def test_ste_vjp_reproduces_soft_vjp(T):
    """With the forward's Viterbi codewords as reference, the STE backward is
    the soft VJP.  Above the precision switch the bits agree.  Below it the
    soft VJP centres on its own fp32 min-sum decode while the STE backward
    takes the exact decode's codewords; any reference gives the same
    gradient, so the two agree to the VJP's tolerance (and bit for bit
    wherever the two decodes pick the same path)."""
    n, k, B, L = 16, 2, 5, 48
    w, c, g = WL.random_case(91, B, L, n)
    wd, cd, gd = dev(w), dev(c), dev(g)
    _, wh = P.viterbi_decode(wd, cd, n, k)
    sdW, sdc = P.bcjr_ste_vjp(wd, cd, n, k, T, wh, gd)
    vdW, vdc = P.bcjr_soft_codeword_vjp(wd, cd, n, k, T, gd)
    torch.cuda.synchronize()
    if T >= 0.04:
        np.testing.assert_array_equal(host(sdW), host(vdW))
        np.testing.assert_array_equal(host(sdc), host(vdc))
    else:
        check_grad(host(vdW), host(sdW).astype(np.float64), "soft vs ste dW")
        check_grad(host(vdc), host(sdc).astype(np.float64), "soft vs ste dc")


def test_ste_vjp_any_reference_same_gradient():
    """The reference only centres the low-temperature tangent: a different
    (finite) reference gives the same gradient to the VJP's tolerance."""
    n, k, B, L, T = 12, 2, 4, 40, 0.01
    w, c, g = WL.random_case(92, B, L, n)
    _, rdW, rdc = O.ste(w, c, n, k, float(np.float32(T)), g)
    dW, dc = P.bcjr_ste_vjp(dev(w), dev(c), n, k, T, dev(w), dev(g))
    torch.cuda.synchronize()
    check_grad(host(dW), rdW, "ref=w dW")
    check_grad(host(dc), rdc, "ref=w dc")


def test_bcjr_quant_matrix_blocks():
    """A weight matrix quantised as row-major blocks of 32: same numbers as the
    [B, L] call, gradient returned in the matrix shape."""
    n, k, T = 10, 2, 0.1
    w, c, g = WL.random_case(93, 8, 96, n)       # 8 x 96 = 24 blocks of 32
    out, dW, dc = autograd_step(w, c, n, k, T, g, hard=True, block=32)
    assert out.shape == w.shape and dW.shape == w.shape
    rwh, rdW, rdc = O.ste(w.reshape(-1, 32), c, n, k, float(np.float32(T)), g.reshape(-1, 32))
    np.testing.assert_array_equal(out.reshape(-1, 32), rwh.astype(np.float32))
    check_grad(dW.reshape(-1, 32), rdW, "matrix dW")
    check_grad(dc, rdc, "matrix dc")


def test_ste_weights_only_gradient():
    """A frozen codebook: only dW is requested and computed."""
    from paper_2605_10655_amd.autograd import BcjrQuant
    n, k, B, L, T = 8, 2, 6, 20, 0.05
    w, c, g = WL.random_case(94, B, L, n)
    wt = dev(w, True)
    out = BcjrQuant.apply(wt, dev(c), n, k, T, True)
    out.backward(dev(g))
    torch.cuda.synchronize()
    _, rdW, _ = O.ste(w, c, n, k, float(np.float32(T)), g, want_dc=False)
    check_grad(host(wt.grad), rdW, "frozen codebook dW")


def test_ste_empty_batch():
    from paper_2605_10655_amd.autograd import BcjrQuant
    wt = torch.empty((0, 8), dtype=torch.float32, device="cuda:0", requires_grad=True)
    ct = dev(np.ones(256, np.float32), True)
    out = BcjrQuant.apply(wt, ct, 8, 2, 0.5, True)
    out.sum().backward()
    torch.cuda.synchronize()
    assert out.shape == (0, 8)
    assert float(ct.grad.abs().max()) == 0.0


def test_ste_full_batch_sampled():
    """The STE step at the benchmark's full size (S = 65536, B = 16384,
    T = 0.05): Viterbi forward and STE backward, checked on sampled blocks."""
    wl = WL.workload(4)
    c, w, g = WL.codebook(4), WL.weights(4), WL.upstream(4)
    n, k, T = wl.state_bits, wl.k, wl.temps[0]
    _say(f"[ste] full batch B={wl.B}")
    wd, cd, gd = dev(w), dev(c), dev(g)
    _, wh = P.viterbi_decode(wd, cd, n, k)
    dW, _ = P.bcjr_ste_vjp(wd, cd, n, k, T, wh, gd, want_dCodebook=False)
    torch.cuda.synchronize()
    idx = WL.parity_subset(4, 6)
    rwh, rdW, _ = O.ste(w[idx], c, n, k, float(np.float32(T)), g[idx], want_dc=False)
    np.testing.assert_array_equal(host(wh)[idx], rwh.astype(np.float32))
    check_grad(host(dW)[idx], rdW, "ste full dW")

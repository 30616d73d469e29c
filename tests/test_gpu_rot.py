"""GPU parity of the rotating in-place exchange kernel (fb_kernel_rot: S =
65536, k = 2, fused w_soft + logZ + dW, T >= 0.04) against the fp64 oracle,
on lengths around the layout's period of 7 steps, L = 1, several
temperatures, the persistent loop and every grid size of a small batch; and
of the dCodebook call at the same shape (which keeps fb_kernel's
two-barrier exchange) on the same cases, against the oracle and against the
rotating kernel.

Tolerances as everywhere: w_soft |err| <= 2e-5, logZ 1e-4 relative, dW 1e-4
of max(|ref_i|, rms(ref)).
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
# (dW, dCodebook also 1e-4 of max(|ref_i|, rms(ref)))
N, KB = 16, 2


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


def fwd_dw(w, c, T, g, workspace=None):
    ws, lz, dW, _ = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), N, KB, T, dev(g), want_dCodebook=False,
                                                 workspace=workspace)
    torch.cuda.synchronize()
    return host(ws), host(lz), host(dW)


def check(w, c, T, g, what):
    ws, lz, dW = fwd_dw(w, c, T, g)
    rws, rlz, rdW, _ = O.soft_codeword_vjp(w, c, N, KB, float(np.float32(T)), g, want_dc=False)
    e = (float(np.abs(ws - rws).max()), float((np.abs(lz - rlz) / np.abs(rlz)).max()), grad_err(dW, rdW))
    _say(f"[rot] {what}: w_soft {e[0]:.2e} logZ {e[1]:.2e} dW {e[2]:.2e}")
    assert np.all(np.isfinite(ws)) and np.all(np.isfinite(dW))
    assert e[0] <= TOL_WS and e[1] <= TOL_LOGZ and e[2] <= TOL_GRAD
    return ws, lz, dW


@pytest.mark.parametrize("L", [1, 2, 6, 7, 8, 13, 15, 22])
@pytest.mark.parametrize("T", [1.0, 0.05])
def test_rotating_exchange_matches_oracle(L, T):
    w, c, g = WL.random_case(9100 + L, 2, L, N)
    check(w, c, T, g, f"L={L} T={T}")


def test_rotating_exchange_config4_blocks_and_dcodebook_kernel():
    """Blocks of the benchmark matrix at T = 0.05 and L = 256 (36 full
    periods of the layout and 4 steps more): against the oracle, and against
    the dCodebook kernel's w_soft, logZ and dW on the same launch."""
    wl = WL.workload(4)
    c = WL.codebook(4)
    w, g = WL.weights(4, rows=2), WL.upstream(4, B=16)
    idx = np.array([0, 5, 11])
    ws, lz, dW = check(w[idx], c, wl.temps[0], g[idx], "cfg4 blocks")
    ws2, lz2, dW2, _ = (host(t) for t in P.bcjr_soft_codeword_fwd_vjp(
        dev(w[idx]), dev(c), N, KB, wl.temps[0], dev(g[idx]), want_dCodebook=True))
    torch.cuda.synchronize()
    assert float(np.abs(ws - ws2).max()) <= TOL_WS
    assert float((np.abs(lz - lz2) / np.abs(lz2)).max()) <= TOL_LOGZ
    assert grad_err(dW, dW2.astype(np.float64)) <= TOL_GRAD


def test_rotating_exchange_every_grid_size():
    """Workspaces of 1 to B slots: grids of 1 to B workgroups, with and
    without the persistent loop, give the same bits."""
    B, L, T = 6, 11, 0.3
    w, c, g = WL.random_case(9300, B, L, N)
    full = check(w, c, T, g, "grid reference")
    big = P.bcjr_workspace_bytes(B, L, N, KB, P.OP_FWD_VJP)
    runs = 0
    for nb in range(1, B + 1):
        size = big * nb // B
        try:
            out = fwd_dw(w, c, T, g, workspace=torch.empty(size, dtype=torch.uint8, device="cuda:0"))
        except P.BcjrError as e:
            assert e.status == -3
            continue
        runs += 1
        for a, b in zip(full, out):
            np.testing.assert_array_equal(a, b)
    _say(f"[rot] {runs} workspace sizes ran")
    assert runs >= B // 2


def fwd_dw_dc(w, c, T, g, workspace=None):
    out = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), N, KB, T, dev(g), want_dCodebook=True,
                                       workspace=workspace)
    torch.cuda.synchronize()
    return tuple(host(t) for t in out)


@pytest.mark.parametrize("L", [1, 6, 7, 15])
@pytest.mark.parametrize("T", [1.0, 0.05])
def test_rotating_exchange_with_dcodebook_matches_oracle(L, T):
    w, c, g = WL.random_case(9500 + L, 3, L, N)
    ws, lz, dW, dc = fwd_dw_dc(w, c, T, g)
    rws, rlz, rdW, rdc = O.soft_codeword_vjp(w, c, N, KB, float(np.float32(T)), g)
    e = (float(np.abs(ws - rws).max()), float((np.abs(lz - rlz) / np.abs(rlz)).max()), grad_err(dW, rdW),
         grad_err(dc, rdc))
    _say(f"[rot dc] L={L} T={T}: w_soft {e[0]:.2e} logZ {e[1]:.2e} dW {e[2]:.2e} dc {e[3]:.2e}")
    assert np.all(np.isfinite(dc))
    assert e[0] <= TOL_WS and e[1] <= TOL_LOGZ and e[2] <= TOL_GRAD and e[3] <= TOL_GRAD
    # the rotating fwd + dW kernel on the same inputs
    ws2, lz2, dW2 = fwd_dw(w, c, T, g)
    assert float(np.abs(ws - ws2).max()) <= TOL_WS
    assert float((np.abs(lz - lz2) / np.abs(lz2)).max()) <= TOL_LOGZ
    assert grad_err(dW2, dW.astype(np.float64)) <= TOL_GRAD


def test_rotating_exchange_with_dcodebook_every_grid_size():
    """dCodebook partials flushed per slot over the persistent loop: every
    grid size gives the same w_soft, logZ and dW bits and the same
    dCodebook up to the order of the fp64 slot sums (one fp32 ulp)."""
    B, L, T = 6, 9, 0.2
    w, c, g = WL.random_case(9600, B, L, N)
    full = fwd_dw_dc(w, c, T, g)
    rws, rlz, rdW, rdc = O.soft_codeword_vjp(w, c, N, KB, float(np.float32(T)), g)
    assert grad_err(full[3], rdc) <= TOL_GRAD and grad_err(full[2], rdW) <= TOL_GRAD
    big = P.bcjr_workspace_bytes(B, L, N, KB, P.OP_FWD_VJP)
    runs = 0
    for nb in range(1, B + 1):
        size = big * nb // B
        try:
            out = fwd_dw_dc(w, c, T, g, workspace=torch.empty(size, dtype=torch.uint8, device="cuda:0"))
        except P.BcjrError as e:
            assert e.status == -3
            continue
        runs += 1
        for a, b in zip(full[:3], out[:3]):
            np.testing.assert_array_equal(a, b)
        a, b = full[3].astype(np.float64), out[3].astype(np.float64)
        assert np.all(np.abs(a - b) <= 2.0 ** -23 * np.abs(a) + 2.0 ** -40 * np.abs(a).max())
    _say(f"[rot dc] {runs} workspace sizes ran")
    assert runs >= B // 2

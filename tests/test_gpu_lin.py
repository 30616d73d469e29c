"""GPU parity of the linear-domain forward-backward kernel (fb_kernel_lin:
S = 65536, k = 2, fused w_soft + logZ + dW, T >= 0.0206) and of its repair
pass: blocks whose group vectors leave the fp32 range are recomputed by the
log-domain kernel (T >= 0.04) or, below, by the double-float kernel centred
on those blocks' decoded codewords.  Batches mix ordinary N(0, 1) blocks with blocks whose
weights sit far outside the codebook (every exponential of a step
underflows, so the block must be marked and recomputed) and blocks with a
few moderate outliers (large single-step decays that the linear kernel
keeps).  Every block is compared with the fp64 oracle.

Tolerances as everywhere: w_soft |err| <= 2e-5, logZ 1e-4 relative, dW 1e-4
of max(|ref_i|, rms(ref)) with the rms over the call's whole output (the
out-of-range blocks have posteriors on one codeword and dW near 1e-30).
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
N, KB = 16, 2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P.load_library()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def grad_err(gpu, ref):
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt(np.mean(ref * ref))
    scale = np.maximum(np.abs(ref), rms)
    return float((np.abs(gpu.astype(np.float64) - ref) / np.where(scale > 0, scale, 1.0)).max())


def mixed_batch(L, seed, far=40.0):
    """Six blocks: 0, 1, 5 N(0, 1); 2 with four weights at +-6 (single-step
    decays of ~40 log2 units at T = 0.05); 3 with every weight at 40 (every
    exponential underflows: marked and recomputed; `far`, 8 in the
    dCodebook tests, is still marked at every temperature tested, and keeps
    (w - c)(X - E X) / T within what the fp32 log-domain repair resolves:
    at 40 that product amplifies the tangents' rounding past the dCodebook
    tolerance, for the log-domain kernels alike); 4 N(0, 1) except one
    weight at 15 mid-block (a single-step decay past the guard at every
    temperature here: marked and recomputed).  Weights further out than
    ~20 from the codebook's range put the local field at thousands of log2
    units, beyond what fp32 log-domain arithmetic resolves to the w_soft
    tolerance; they are outside this test."""
    r = np.random.Generator(np.random.PCG64(seed))
    w = r.standard_normal((6, L)).astype(np.float32)
    if L >= 4:
        w[2, [0, L // 3, L // 2, L - 1]] = [6.0, -6.0, 6.0, -6.0]
    else:
        w[2, 0] = 6.0
    w[3, :] = far
    w[4, L // 2] = 15.0
    g = r.standard_normal((6, L)).astype(np.float32)
    return w, g


@pytest.mark.parametrize("T", [0.021, 0.03, 0.05, 0.1, 1.0])
@pytest.mark.parametrize("L", [1, 9, 256])
def test_linear_kernel_and_repair_pass_match_oracle(L, T):
    c = WL.codebook(4)
    w, g = mixed_batch(L, 4100 + L)
    print(f"linear kernel: L={L} T={T} B=6 (mixed, with out-of-range blocks)", flush=True)
    ws, lz, dW, _ = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), N, KB, T, dev(g), want_dCodebook=False)
    torch.cuda.synchronize()
    rws, rlz, rdW, _ = O.soft_codeword_vjp(w, c, N, KB, float(np.float32(T)), g, want_dc=False)
    ws, lz, dW = ws.cpu().numpy(), lz.cpu().numpy(), dW.cpu().numpy()
    assert np.isfinite(ws).all() and np.isfinite(lz).all() and np.isfinite(dW).all()
    e_ws = float(np.abs(ws - rws).max())
    e_lz = float((np.abs(lz - rlz) / np.abs(rlz)).max())
    e_dw = grad_err(dW, rdW)
    print(f"  w_soft {e_ws:.2e} logZ {e_lz:.2e} dW {e_dw:.2e}", flush=True)
    assert e_ws <= TOL_WS and e_lz <= TOL_LOGZ and e_dw <= TOL_GRAD


@pytest.mark.parametrize("T", [0.021, 0.05])
def test_repair_pass_under_every_grid_size(T):
    """Under every workspace size from one slot up (grids of one workgroup,
    which then walks every block in the same slot, to one per block) the
    out-of-range blocks are recomputed and the result is the same bits as
    with a full workspace; the full-size run matches the oracle."""
    c = WL.codebook(4)
    L = 24
    w, g = mixed_batch(L, 4200)
    B = w.shape[0]
    print(f"linear kernel grids: L={L} T={T} B={B}", flush=True)

    def run(work=None):
        out = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), N, KB, T, dev(g), want_dCodebook=False,
                                           workspace=work)
        torch.cuda.synchronize()
        return [x.cpu().numpy() for x in out[:3]]

    full = run()
    rws, rlz, rdW, _ = O.soft_codeword_vjp(w, c, N, KB, float(np.float32(T)), g, want_dc=False)
    assert float(np.abs(full[0] - rws).max()) <= TOL_WS
    assert float((np.abs(full[1] - rlz) / np.abs(rlz)).max()) <= TOL_LOGZ
    assert grad_err(full[2], rdW) <= TOL_GRAD
    big = P.bcjr_workspace_bytes(B, L, N, KB, P.OP_FWD_VJP)
    runs = 0
    for nb in range(1, B + 1):
        size = big * nb // B
        try:
            out = run(torch.empty(size, dtype=torch.uint8, device="cuda:0"))
        except P.BcjrError as e:
            assert e.status == -3
            continue
        runs += 1
        for a, b in zip(out, full):
            assert np.array_equal(a, b)
    print(f"  {runs} workspace sizes ran", flush=True)
    assert runs >= 2


@pytest.mark.parametrize("T", [0.021, 0.0268])
def test_linear_kernel_low_temperature_full_batch_sampled(T):
    """The q/o-projection matrix (16384 blocks of 256, S = 65536) below the
    log-domain kernel's range (T = 0.0268 is the third of the 8 annealed
    temperatures): sampled blocks against the oracle."""
    W, C, G = WL.weights(4), WL.codebook(4), WL.upstream(4)
    print(f"linear kernel full batch: B={W.shape[0]} T={T}", flush=True)
    ws, lz, dW, _ = P.bcjr_soft_codeword_fwd_vjp(dev(W), dev(C), N, KB, T, dev(G), want_dCodebook=False)
    torch.cuda.synchronize()
    idx = WL.parity_subset(4, 16)
    rws, rlz, rdW, _ = O.soft_codeword_vjp(W[idx], C, N, KB, float(np.float32(T)), G[idx], want_dc=False)
    ws, lz, dW = ws.cpu().numpy()[idx], lz.cpu().numpy()[idx], dW.cpu().numpy()[idx]
    e_ws = float(np.abs(ws - rws).max())
    e_lz = float((np.abs(lz - rlz) / np.abs(rlz)).max())
    e_dw = grad_err(dW, rdW)
    print(f"  w_soft {e_ws:.2e} logZ {e_lz:.2e} dW {e_dw:.2e}", flush=True)
    assert e_ws <= TOL_WS and e_lz <= TOL_LOGZ and e_dw <= TOL_GRAD


@pytest.mark.parametrize("T", [0.021, 0.05, 1.0])
@pytest.mark.parametrize("L", [1, 9, 256])
def test_linear_soft_codeword_and_repair_match_oracle(L, T):
    """bcjr_soft_codeword (w_soft and logZ alone) through the linear kernel's
    soft-codeword form, with the out-of-range blocks of the mixed batch
    recomputed by the log-domain soft-codeword kernel."""
    c = WL.codebook(4)
    w, _ = mixed_batch(L, 4500 + L)
    print(f"linear soft codeword: L={L} T={T} B=6 (mixed)", flush=True)
    ws, lz = P.bcjr_soft_codeword(dev(w), dev(c), N, KB, T)
    torch.cuda.synchronize()
    rws, rlz = O.soft_codeword(w, c, N, KB, float(np.float32(T)))
    ws, lz = ws.cpu().numpy(), lz.cpu().numpy()
    assert np.isfinite(ws).all() and np.isfinite(lz).all()
    e_ws = float(np.abs(ws - rws).max())
    e_lz = float((np.abs(lz - rlz) / np.abs(rlz)).max())
    print(f"  w_soft {e_ws:.2e} logZ {e_lz:.2e}", flush=True)
    assert e_ws <= TOL_WS and e_lz <= TOL_LOGZ


def test_linear_soft_codeword_every_grid_size():
    """The soft-codeword form under every workspace size from one slot up:
    the same bits as with a full workspace, out-of-range blocks included."""
    c = WL.codebook(4)
    L, T = 24, 0.05
    w, _ = mixed_batch(L, 4600)
    B = w.shape[0]

    def run(work=None):
        out = P.bcjr_soft_codeword(dev(w), dev(c), N, KB, T, workspace=work)
        torch.cuda.synchronize()
        return [x.cpu().numpy() for x in out]

    full = run()
    rws, rlz = O.soft_codeword(w, c, N, KB, float(np.float32(T)))
    assert float(np.abs(full[0] - rws).max()) <= TOL_WS
    big = P.bcjr_workspace_bytes(B, L, N, KB, P.OP_FWD)
    runs = 0
    for nb in range(1, B + 1):
        try:
            out = run(torch.empty(big * nb // B, dtype=torch.uint8, device="cuda:0"))
        except P.BcjrError as e:
            assert e.status == -3
            continue
        runs += 1
        for a, b in zip(out, full):
            assert np.array_equal(a, b)
    print(f"linear soft codeword grids: {runs} workspace sizes ran", flush=True)
    assert runs >= 2


def test_linear_soft_codeword_full_batch_sampled():
    """bcjr_soft_codeword on the q/o-projection matrix at T = 0.05: sampled
    blocks against the oracle."""
    W, C = WL.weights(4), WL.codebook(4)
    ws, lz = P.bcjr_soft_codeword(dev(W), dev(C), N, KB, 0.05)
    torch.cuda.synchronize()
    idx = WL.parity_subset(4, 16)
    rws, rlz = O.soft_codeword(W[idx], C, N, KB, float(np.float32(0.05)))
    e_ws = float(np.abs(ws.cpu().numpy()[idx] - rws).max())
    e_lz = float((np.abs(lz.cpu().numpy()[idx] - rlz) / np.abs(rlz)).max())
    print(f"linear soft codeword full batch: w_soft {e_ws:.2e} logZ {e_lz:.2e}", flush=True)
    assert e_ws <= TOL_WS and e_lz <= TOL_LOGZ


@pytest.mark.parametrize("L,T", [(2048, 0.05), (2048, 0.021), (64, 25.0)])
def test_linear_kernel_long_blocks_and_high_temperature(L, T):
    """Long blocks (the tracked exponents of the rescales reach thousands)
    and a temperature at which every step's vector grows: fwd + dW and the
    soft codeword alone against the oracle."""
    c = WL.codebook(4)
    r = np.random.Generator(np.random.PCG64(4700 + L))
    w = r.standard_normal((2, L)).astype(np.float32)
    g = r.standard_normal((2, L)).astype(np.float32)
    print(f"linear kernel: L={L} T={T} B=2", flush=True)
    ws, lz, dW, _ = P.bcjr_soft_codeword_fwd_vjp(dev(w), dev(c), N, KB, T, dev(g), want_dCodebook=False)
    ss, sl = P.bcjr_soft_codeword(dev(w), dev(c), N, KB, T)
    torch.cuda.synchronize()
    rws, rlz, rdW, _ = O.soft_codeword_vjp(w, c, N, KB, float(np.float32(T)), g, want_dc=False)
    ws, lz, dW, ss, sl = (x.cpu().numpy() for x in (ws, lz, dW, ss, sl))
    e_ws = max(float(np.abs(ws - rws).max()), float(np.abs(ss - rws).max()))
    e_lz = max(float((np.abs(lz - rlz) / np.abs(rlz)).max()), float((np.abs(sl - rlz) / np.abs(rlz)).max()))
    e_dw = grad_err(dW, rdW)
    print(f"  w_soft {e_ws:.2e} logZ {e_lz:.2e} dW {e_dw:.2e}", flush=True)
    assert e_ws <= TOL_WS and e_lz <= TOL_LOGZ and e_dw <= TOL_GRAD

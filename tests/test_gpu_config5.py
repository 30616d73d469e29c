"""Parity at the annealed gate/up-projection workload's production shape:
the 2048 x 8192 N(0,1) matrix as 65536 blocks of L = 256, S = 65536, k = 2,
fused w_soft + logZ + dW + dCodebook in ONE launch over all blocks (the
launch the annealed-calls benchmark times: 256 persistent workgroups, each
walking 256 blocks through its workspace slot).

Checked per call:
  * sampled blocks against the fp64 oracle (w_soft |err| <= 2e-5, logZ
    1e-4 relative, dW 1e-4 of max(|ref|, rms(ref)));
  * the same sampled blocks launched on their own (one block per
    workgroup): every per-block output is bit-identical, since a block's
    arithmetic does not depend on the slot or the loop iteration it runs in;
  * dCodebook, a sum over all 65536 blocks, against the sum of two launches
    over the two halves of the matrix (the fp64 per-slot partials are
    summed in another order and rounded to fp32 once per launch, so the
    difference is a few fp32 roundings of the summands' size);
  * the same blocks' dCodebook as its own launch against the oracle.
The last call (T = 0.001) is also checked against the Viterbi decode (the
T -> 0 limit of Sec. 3.3): wherever the oracle's min-sum max-marginal energy
gap exceeds T ln(max|c_i - c_j| / 2e-5), the soft codeword must equal the
decoded codeword within 2e-5; the positions below that gap are counted and
reported, not checked.
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
TOL_LOGZ = 1e-4
TOL_GRAD = 1e-4


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def cfg5():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P.load_library()
    wl = WL.workload(5)
    d = torch.device("cuda:0")
    w = WL.weights(5)
    c = WL.codebook(5)
    ws_bytes = P.bcjr_workspace_bytes(wl.B, wl.L, wl.state_bits, wl.k, P.OP_FWD_VJP)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=d)
    yield wl, w, c, torch.from_numpy(w).to(d), torch.from_numpy(c).to(d), ws
    del ws
    torch.cuda.empty_cache()


def host(t):
    return t.detach().cpu().numpy()


def grad_err(gpu, ref):
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt(np.mean(ref * ref))
    scale = np.maximum(np.abs(ref), rms)
    return float((np.abs(gpu.astype(np.float64) - ref) / np.where(scale > 0, scale, 1.0)).max())


def launch(wd, cd, n, k, T, gd, ws=None):
    out = P.bcjr_soft_codeword_fwd_vjp(wd, cd, n, k, T, gd, workspace=ws)
    torch.cuda.synchronize()
    return tuple(host(t) for t in out)


@pytest.mark.parametrize("call", [7, 1])
def test_production_launch_all_blocks(cfg5, call):
    wl, w, c, wd, cd, ws = cfg5
    n, k = wl.state_bits, wl.k
    T = wl.temps[call]
    g = WL.upstream(5, call=call)
    gd = torch.from_numpy(g).to(wd.device)
    _say(f"[cfg5] call {call} T={T:.4g}: one launch over B={wl.B} blocks (w_soft, logZ, dW, dc)")
    fws, flz, fdW, fdc = launch(wd, cd, n, k, T, gd, ws)
    for name, a in (("w_soft", fws), ("logZ", flz), ("dW", fdW), ("dc", fdc)):
        assert np.all(np.isfinite(a)), f"non-finite {name}"

    # sampled blocks against the oracle
    idx = WL.parity_subset(5, 8)
    _say(f"[cfg5] call {call}: oracle on blocks {idx.tolist()}")
    rws, rlz, rdW, _ = O.soft_codeword_vjp(w[idx], c, n, k, float(np.float32(T)), g[idx],
                                           want_dc=False)
    e_ws = float(np.abs(fws[idx] - rws).max())
    e_lz = float((np.abs(flz[idx] - rlz) / np.abs(rlz)).max())
    e_dw = grad_err(fdW[idx], rdW)
    _say(f"[cfg5] call {call}: w_soft {e_ws:.2e} logZ {e_lz:.2e} dW {e_dw:.2e}")
    assert e_ws <= TOL_WS and e_lz <= TOL_LOGZ and e_dw <= TOL_GRAD

    # the same blocks as their own launch: bit-identical per-block outputs;
    # their dCodebook against the oracle
    sws, slz, sdW, sdc = launch(torch.from_numpy(w[idx]).to(wd.device), cd, n, k, T,
                                torch.from_numpy(g[idx]).to(wd.device))
    np.testing.assert_array_equal(sws, fws[idx])
    np.testing.assert_array_equal(slz, flz[idx])
    np.testing.assert_array_equal(sdW, fdW[idx])
    rdc = O.soft_codeword_vjp(w[idx], c, n, k, float(np.float32(T)), g[idx])[3]
    e_dc = grad_err(sdc, rdc)
    _say(f"[cfg5] call {call}: subset launch bit-identical; its dc {e_dc:.2e}")
    assert e_dc <= TOL_GRAD

    # dCodebook over all blocks = the two halves' dCodebook
    h = wl.B // 2
    dca = launch(wd[:h], cd, n, k, T, gd[:h], ws)[3].astype(np.float64)
    dcb = launch(wd[h:], cd, n, k, T, gd[h:], ws)[3].astype(np.float64)
    scale = np.abs(dca) + np.abs(dcb) + np.abs(fdc.astype(np.float64))
    dev = np.abs(fdc - (dca + dcb)) / np.maximum(scale, 1e-30)
    _say(f"[cfg5] call {call}: dc vs halves max rel dev {dev.max():.2e}")
    assert dev.max() <= 4 * 2.0 ** -24
    # translation invariance of the whole launch: sum dW + sum dc = sum g
    # (every block contributes sum_t g_t - sum_t dW_t to sum dc)
    lhs = fdW.astype(np.float64).sum() + fdc.astype(np.float64).sum()
    rhs = g.astype(np.float64).sum()
    _say(f"[cfg5] call {call}: sum dW + sum dc = {lhs:.6f}, sum g = {rhs:.6f}")
    assert abs(lhs - rhs) <= 1e-4 * (np.abs(fdW).astype(np.float64).sum()
                                     + np.abs(fdc).astype(np.float64).sum())

    if call == len(wl.temps) - 1:
        _say(f"[cfg5] final call: Viterbi decode of all {wl.B} blocks")
        st, wh = P.viterbi_decode(wd, cd, n, k)
        torch.cuda.synchronize()
        st, wh = host(st), host(wh)
        np.testing.assert_array_equal(wh, c[st])
        rst, _ = O.viterbi(w[idx], c, n, k)
        np.testing.assert_array_equal(st[idx], rst)
        held, gap, thr = O.crisp_positions(w[idx], c, n, k, float(np.float32(T)), rst)
        dev = np.abs(fws[idx].astype(np.float64) - c[rst])
        excused = int((~held).sum())
        _say(f"[cfg5] final call: gap threshold {thr:.4g}; {excused} of {held.size} sampled "
              f"positions excused (gap below it); max |w_soft - c(s*)| on the rest "
              f"{dev[held].max():.2e}; all blocks within 2e-5 of c(s*): "
              f"{float((np.abs(fws - wh) <= 2e-5).mean()):.4f}")
        assert held.mean() > 0.8
        assert dev[held].max() <= TOL_WS

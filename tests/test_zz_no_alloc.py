"""bcjr_soft_codeword_fwd_vjp_noalloc, called through the C ABI (ctypes, raw
device pointers, caller-allocated outputs), against
bcjr_soft_codeword_fwd_vjp with its own workspace.

The two calls run the same kernels with different workspaces and so with
different grids; a block's arithmetic does not depend on the slot it runs
in, so w_soft, logZ and dW must agree bit for bit, and dCodebook (fp64
per-slot partials, or fp64 atomic sums on the pruned low-temperature path,
added in another order, then rounded to fp32 once) to a few fp32 roundings.  Two calls in a row share the GPU's one scratch array:
the second, smaller call (another trellis size, the double-float
low-temperature kernel and its reference decode) must not see the first
call's leftovers.  A shape whose single block slot exceeds the array is
refused with BCJR_ERR_WORKSPACE before any launch.
"""
import ctypes
import sys

import numpy as np
import pytest

import paper_2605_10655_amd as P
from paper_2605_10655_amd import workloads as WL

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return P.load_library()


def _p(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _noalloc(lib, w, c, n, k, T, g, want_dc=True):
    d = torch.device("cuda:0")
    wd, cd, gd = (torch.from_numpy(a).to(d) for a in (w, c, g))
    B, L = w.shape
    ws, dW = torch.empty_like(wd), torch.empty_like(wd)
    lz = torch.empty(B, dtype=torch.float32, device=d)
    dc = torch.full_like(cd, np.nan) if want_dc else None
    stream = torch.cuda.current_stream()
    rc = lib.bcjr_soft_codeword_fwd_vjp_noalloc(_p(wd), B, L, _p(cd), n, k, float(T), _p(gd), _p(ws),
                                                _p(lz), _p(dW), _p(dc),
                                                ctypes.c_void_p(stream.cuda_stream))
    assert rc == 0, P.bcjr_status_string(rc)
    torch.cuda.synchronize()
    return tuple(None if t is None else t.cpu().numpy() for t in (ws, lz, dW, dc))


def _reference(w, c, n, k, T, g, want_dc=True):
    d = torch.device("cuda:0")
    out = P.bcjr_soft_codeword_fwd_vjp(*(torch.from_numpy(a).to(d) for a in (w, c)), n, k, T,
                                       torch.from_numpy(g).to(d), want_dCodebook=want_dc)
    torch.cuda.synchronize()
    return tuple(None if t is None else t.cpu().numpy() for t in out)


def _compare(got, ref, what):
    for name, a, b in zip(("w_soft", "logZ", "dW"), got[:3], ref[:3]):
        np.testing.assert_array_equal(a, b, err_msg=f"{what}: {name}")
    if got[3] is None:
        assert ref[3] is None
        _say(f"[noalloc] {what}: outputs bit-identical")
        return
    a, b = got[3].astype(np.float64), ref[3].astype(np.float64)
    dev = np.abs(a - b) / np.maximum(np.abs(a) + np.abs(b), 1e-30)
    _say(f"[noalloc] {what}: per-block outputs bit-identical; dc max rel dev {dev.max():.2e}")
    assert np.all(np.isfinite(a)) and dev.max() <= 4 * 2.0 ** -24


def test_noalloc_matches_workspace_entry_point_on_two_calls(lib):
    # first call: the S = 65536 fp32 kernel with dCodebook; the scratch holds
    # 20 of its 12.5 MiB block slots, so four workgroups run a second block
    # (the workspace call runs one block per workgroup)
    w, c, g = WL.random_case(9001, 24, 48, 16)
    _say("[noalloc] call 1: n=16 k=2 B=24 L=48 T=0.05")
    _compare(_noalloc(lib, w, c, 16, 2, 0.05, g), _reference(w, c, 16, 2, 0.05, g), "call 1")
    # second, smaller call on the same scratch: another trellis and the
    # double-float kernel, whose reference decode also lives in the scratch
    w2, c2, g2 = WL.random_case(9002, 7, 20, 12)
    _say("[noalloc] call 2: n=12 k=2 B=7 L=20 T=0.003")
    _compare(_noalloc(lib, w2, c2, 12, 2, 0.003, g2), _reference(w2, c2, 12, 2, 0.003, g2),
             "call 2")
    # third: S = 65536 without dCodebook, the rotating-exchange kernel
    w3, c3, g3 = WL.random_case(9003, 5, 16, 16)
    _say("[noalloc] call 3: n=16 k=2 B=5 L=16 T=0.1, no dCodebook")
    _compare(_noalloc(lib, w3, c3, 16, 2, 0.1, g3, want_dc=False),
             _reference(w3, c3, 16, 2, 0.1, g3, want_dc=False), "call 3")
    # fourth: S = 65536 at T = 0.008, the pruned kernels (min-sum sweeps,
    # kept-state bitmaps and fp64 entries in the scratch, dCodebook through
    # an fp64 accumulator there)
    w4, c4, g4 = WL.random_case(9004, 5, 32, 16)
    _say("[noalloc] call 4: n=16 k=2 B=5 L=32 T=0.008")
    _compare(_noalloc(lib, w4, c4, 16, 2, 0.008, g4), _reference(w4, c4, 16, 2, 0.008, g4), "call 4")


def test_noalloc_refuses_a_slot_larger_than_the_scratch(lib):
    # one block at S = 65536 with L = 10000: its fp32 history alone is
    # 10000 x 2 x 16384 x 4 B = 1.3 GB, beyond the 256 MiB array
    d = torch.device("cuda:0")
    B, L, n, k = 1, 10000, 16, 2
    w = torch.zeros((B, L), dtype=torch.float32, device=d)
    c = torch.zeros(1 << n, dtype=torch.float32, device=d)
    ws = torch.empty_like(w)
    rc = lib.bcjr_soft_codeword_fwd_vjp_noalloc(_p(w), B, L, _p(c), n, k, 0.05, _p(w), _p(ws),
                                                _p(None), _p(None), _p(None),
                                                ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == -3, P.bcjr_status_string(rc)

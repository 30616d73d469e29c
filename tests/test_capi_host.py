"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function declared in include/bcjr.h,
size workspaces by pure host arithmetic, and reject bad arguments before
touching the device.  No call here reaches a kernel launch.
"""
import ctypes
import os
import re

import pytest

import paper_2605_10655_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bcjr.h")

FAKE = 1 << 20          # 16-byte aligned non-null address, never dereferenced
MISALIGNED = FAKE + 4


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"if", "sizeof"})


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(P.library_path()):
        pytest.skip("libbcjr.so not built")
    return P.load_library()


def test_library_exports_every_declared_function(lib):
    names = header_functions()
    assert set(names) >= {"bcjr_workspace_bytes", "bcjr_soft_codeword", "bcjr_soft_codeword_vjp",
                          "bcjr_soft_codeword_fwd_vjp", "bcjr_ste_vjp", "viterbi_decode",
                          "bcjr_status_string"}
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4):
        assert P.bcjr_status_string(code)
    assert P.bcjr_status_string(12345) == "unknown status"


def test_workspace_bytes_host_arithmetic(lib):
    ws = P.bcjr_workspace_bytes
    # invalid / unsupported / empty
    assert ws(10, 0, 4, 2, P.OP_FWD) == 0
    assert ws(10, 16, 4, 5, P.OP_FWD) == 0
    assert ws(10, 16, 17, 2, P.OP_FWD) == 0
    assert ws(10, 16, 4, 2, P.OP_FWD) > 0
    assert ws(0, 16, 4, 2, P.OP_FWD) == 0
    assert ws(10, 16, 4, 2, 9) == 0
    # supported shapes give positive sizes that grow with L and with the VJP
    for n, k in [(4, 2), (8, 2), (12, 2), (16, 2), (2, 1), (14, 1), (6, 3), (14, 3)]:
        f = ws(100, 32, n, k, P.OP_FWD)
        v = ws(100, 32, n, k, P.OP_FWD_VJP)
        assert 0 < f < v
        assert ws(100, 64, n, k, P.OP_FWD) > f
        assert ws(100, 32, n, k, P.OP_VITERBI) > 0
    # every 1 <= k <= n <= 16: the super-group families, or the fp64 generic
    # family (n < 2k, k >= 4, k = 1 at 15-16 bits, k = 3 above 14)
    for n in range(1, 17):
        for k in range(1, n + 1):
            for op in (P.OP_FWD, P.OP_VJP, P.OP_FWD_VJP, P.OP_VITERBI):
                assert ws(4, 8, n, k, op) > 0, (n, k, op)
    # generic family: H and B histories of L x S/K doubles, four group
    # vectors, the S-entry dCodebook partial, per slot; one slot per block here
    L, n, k = 8, 6, 4
    assert ws(3, L, n, k, P.OP_FWD_VJP) == 3 * 8 * (2 * L * 4 + 4 * 4 + 64)
    assert ws(3, L, n, k, P.OP_FWD) == 3 * 8 * (L * 4 + 4 * 4)
    assert ws(3, L, n, k, P.OP_VITERBI) == 3 * (2 * 4 * 8 + L * 4 * 2)
    assert ws(1, (1 << 30) + 1, 3, 2, P.OP_FWD) == 0   # generic family: L up to 2^30
    # 32-bit history offsets: one workgroup's histories below 2 GiB
    assert ws(4, 16383, 16, 2, P.OP_FWD) > 0
    assert ws(4, 16383, 16, 2, P.OP_VITERBI) > 0
    assert ws(4, 16384, 16, 2, P.OP_FWD) == 0
    assert ws(4, 16384, 16, 2, P.OP_VITERBI) == 0
    assert ws(4, 10922, 16, 2, P.OP_FWD_VJP) > 0
    assert ws(4, 10923, 16, 2, P.OP_FWD_VJP) == 0
    for n, k in [(4, 2), (8, 2), (12, 2), (16, 2), (2, 1), (14, 1), (6, 3), (14, 3)]:
        assert ws(4, 16383, n, k, P.OP_FWD) > 0, (n, k)
        assert ws(4, 10922, n, k, P.OP_FWD_VJP) > 0, (n, k)
    # the S = 65536 histories: per block L * S/K * (4 + 8) bytes plus small arrays
    B, L = 16384, 256
    per_slot = L * (1 << 14) * 12
    assert ws(B, L, 16, 2, P.OP_FWD_VJP) >= 256 * per_slot


def _soft(lib, w=FAKE, B=4, L=8, c=FAKE, n=4, k=2, T=1.0, out=FAKE, lz=None, ws=None, wsb=0):
    return lib.bcjr_soft_codeword(w, B, L, c, n, k, T, out, lz, ws, wsb, None)


def test_soft_codeword_argument_validation(lib):
    E = -1
    assert _soft(lib, B=-1) == E
    assert _soft(lib, L=0) == E
    assert _soft(lib, k=0) == E
    assert _soft(lib, n=1, k=2) == E
    assert _soft(lib, n=17) == E
    assert _soft(lib, T=0.0) == E
    assert _soft(lib, T=-1.0) == E
    assert _soft(lib, T=float("nan")) == E
    assert _soft(lib, T=float("inf")) == E
    assert _soft(lib, w=None) == E
    assert _soft(lib, c=None) == E
    assert _soft(lib, out=None) == E
    assert _soft(lib, c=MISALIGNED) == E
    assert _soft(lib, w=FAKE + 2) == E
    assert _soft(lib, n=3, k=2) == -3                 # generic family: needs a workspace
    assert _soft(lib, n=16, k=1) == -3
    assert _soft(lib, n=16, k=4) == -3
    assert _soft(lib, n=3, k=2, L=(1 << 30) + 1) == -2  # beyond the generic family's L
    assert _soft(lib, n=16, k=2, L=16384) == -2       # history offsets past 2^31 bytes
    assert _soft(lib, ws=None) == -3                  # no workspace
    assert _soft(lib, ws=FAKE + 8, wsb=1 << 20) == -3  # misaligned workspace
    assert _soft(lib, B=0) == 0                       # empty batch is a no-op


def test_vjp_and_viterbi_argument_validation(lib):
    f = lib.bcjr_soft_codeword_fwd_vjp
    assert f(FAKE, 4, 8, FAKE, 4, 2, 1.0, None, FAKE, None, None, None, None, 0, None) == -1
    assert f(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE + 1, FAKE, None, None, None, None, 0, None) == -1
    assert f(FAKE, 4, 8, FAKE, 4, 2, 0.0, FAKE, FAKE, None, None, None, None, 0, None) == -1
    assert f(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE, FAKE, None, FAKE, None, None, 0, None) == -3
    assert f(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE, None, None, None, None, None, 0, None) == 0
    assert f(FAKE, 0, 8, FAKE, 4, 2, 1.0, FAKE, None, None, None, None, None, 0, None) == 0
    v = lib.bcjr_soft_codeword_vjp
    assert v(FAKE, 4, 8, FAKE, 4, 2, 1.0, None, FAKE, None, None, 0, None) == -1
    assert v(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE, None, None, None, 0, None) == 0
    st = lib.bcjr_ste_vjp
    assert st(FAKE, 4, 8, FAKE, 4, 2, 1.0, None, FAKE, FAKE, None, None, 0, None) == -1  # w_hard
    assert st(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE + 2, FAKE, FAKE, None, None, 0, None) == -1
    assert st(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE, None, FAKE, None, None, 0, None) == -1  # grad
    assert st(FAKE, 4, 8, FAKE, 4, 2, -1.0, FAKE, FAKE, FAKE, None, None, 0, None) == -1
    assert st(FAKE, 4, (1 << 30) + 1, FAKE, 3, 2, 1.0, FAKE, FAKE, FAKE, None, None, 0, None) == -2
    assert st(FAKE, 4, 8, FAKE, 3, 2, 1.0, FAKE, FAKE, FAKE, None, None, 0, None) == -3
    assert st(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE, FAKE, FAKE, None, None, 0, None) == -3
    assert st(FAKE, 4, 8, FAKE, 4, 2, 1.0, FAKE, FAKE, None, None, None, 0, None) == 0
    assert st(FAKE, 0, 8, FAKE, 4, 2, 1.0, None, None, None, None, None, 0, None) == 0
    vd = lib.viterbi_decode
    assert vd(FAKE, 4, 8, FAKE, 4, 2, None, None, FAKE, 1 << 20, None) == -1
    assert vd(FAKE, 4, 8, FAKE, 4, 2, FAKE, None, None, 0, None) == -3
    assert vd(FAKE, 4, (1 << 30) + 1, FAKE, 3, 2, FAKE, None, FAKE, 1 << 20, None) == -2
    assert vd(FAKE, 0, 8, FAKE, 4, 2, FAKE, None, None, 0, None) == 0


def test_python_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    """No silent fallback: a missing library is an ImportError."""
    monkeypatch.setattr(P, "_lib", None)
    monkeypatch.setattr(P, "library_path", lambda: str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        P.load_library()


def test_autograd_layer_refuses_host_tensors(lib):
    """The autograd node has no CPU path: host tensors are an error."""
    torch = pytest.importorskip("torch")
    from paper_2605_10655_amd.autograd import BcjrQuant, bcjr_quant
    w = torch.zeros(2, 8, requires_grad=True)
    c = torch.zeros(16)
    for hard in (False, True):
        with pytest.raises(TypeError):
            BcjrQuant.apply(w, c, 4, 2, 0.5, hard)
    with pytest.raises(ValueError):
        bcjr_quant(torch.zeros(3, 5), c, 4, 2, 0.5, block=4)


def test_vector_emission_host_checks(lib):
    ws = P.bcjr_vec_workspace_bytes
    assert ws(16, 256, 16, 4, 2, P.OP_FWD) > 0
    assert ws(16, 256, 16, 4, 2, P.OP_VJP) > ws(16, 256, 16, 4, 2, P.OP_FWD)
    assert ws(16, 256, 16, 4, 2, P.OP_VITERBI) > 0
    assert ws(16, 255, 16, 4, 2, P.OP_FWD) == 0          # L not a multiple of V
    assert ws(16, 256, 16, 2, 2, P.OP_FWD) == 0          # only k = 4 with V = 2
    assert ws(16, 256, 7, 4, 2, P.OP_FWD) == 0           # state_bits >= 8
    assert ws(16, 256, 16, 4, 3, P.OP_FWD) == 0
    assert ws(16, 256, 16, 2, 1, P.OP_FWD) == P.bcjr_workspace_bytes(16, 256, 16, 2, P.OP_FWD)
    # 32-bit history offsets: N = L / 2 steps, 16 bytes per group with the VJP
    assert ws(4, 2 * 32767, 16, 4, 2, P.OP_FWD_VJP) > 0
    assert ws(4, 2 * 32768, 16, 4, 2, P.OP_FWD_VJP) == 0
    assert ws(4, 2 * 131071, 16, 4, 2, P.OP_FWD) > 0
    f = lib.bcjr_vec_soft_codeword
    assert f(FAKE, 4, 8, FAKE, 8, 4, 2, 1.0, FAKE, None, None, 0, None) == -3
    assert f(FAKE, 4, 7, FAKE, 8, 4, 2, 1.0, FAKE, None, None, 0, None) == -1  # L % V
    assert f(FAKE, 4, 8, FAKE, 8, 4, 2, 0.0, FAKE, None, None, 0, None) == -1
    assert f(FAKE, 4, 8, FAKE, 8, 3, 2, 1.0, FAKE, None, None, 0, None) == -2
    assert f(FAKE, 4, 8, MISALIGNED, 8, 4, 2, 1.0, FAKE, None, None, 0, None) == -1
    assert f(FAKE, 0, 8, FAKE, 8, 4, 2, 1.0, FAKE, None, None, 0, None) == 0
    v = lib.bcjr_vec_soft_codeword_fwd_vjp
    assert v(FAKE, 4, 8, FAKE, 8, 4, 2, 0.03, FAKE, FAKE, None, None, None, None, 0, None) == -3
    assert v(FAKE, 4, 8, FAKE, 8, 4, 2, 0.5, None, FAKE, None, None, None, None, 0, None) == -1
    assert v(FAKE, 4, 8, FAKE, 8, 4, 2, 0.5, FAKE, FAKE, None, None, None, None, 0, None) == -3
    vd = lib.bcjr_vec_viterbi_decode
    assert vd(FAKE, 4, 8, FAKE, 8, 4, 2, None, None, FAKE, 1 << 20, None) == -1
    assert vd(FAKE, 4, 8, FAKE, 8, 4, 2, FAKE, None, None, 0, None) == -3
    assert vd(FAKE, 0, 8, FAKE, 8, 4, 2, None, None, None, 0, None) == 0


def test_training_helpers_argument_validation(lib):
    g = lib.bcjr_gaussian_codebook
    assert g(None, 8, 1, 0, None) == -1
    assert g(FAKE, 0, 1, 0, None) == -1
    assert g(FAKE, 25, 1, 0, None) == -1
    assert g(FAKE, 8, 9, 0, None) == -1
    assert g(FAKE + 2, 8, 1, 0, None) == -1
    a = lib.qat_adam_step
    assert a(None, None, None, None, 0, 1e-3, 0.9, 0.999, 1e-8, 1, 0.0, None) == 0  # empty
    assert a(FAKE, FAKE, FAKE, FAKE, 4, 1e-3, 0.9, 0.999, 1e-8, 0, 0.0, None) == -1  # step 0
    assert a(FAKE, FAKE, FAKE, FAKE, 4, 1e-3, 1.0, 0.999, 1e-8, 1, 0.0, None) == -1  # beta1
    assert a(FAKE, FAKE, FAKE, FAKE, 4, 1e-3, 0.9, 0.999, 0.0, 1, 0.0, None) == -1   # eps
    assert a(FAKE, None, FAKE, FAKE, 4, 1e-3, 0.9, 0.999, 1e-8, 1, 0.0, None) == -1
    s = lib.qat_sgd_step
    assert s(None, None, 0, 0.1, 0.0, None) == 0
    assert s(FAKE, FAKE, 4, -0.1, 0.0, None) == -1
    assert s(FAKE, FAKE, 4, 0.1, -1.0, None) == -1


def test_ldlq_argument_validation(lib):
    import ctypes as C
    L = lib
    L.bcjr_block_ldl_workspace_bytes.argtypes = [C.c_int64, C.c_int64]
    L.bcjr_block_ldl_workspace_bytes.restype = C.c_size_t
    L.bcjr_block_ldl.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_double, C.c_void_p, C.c_void_p,
                                 C.c_void_p, C.c_size_t, C.c_void_p]
    L.bcjr_ldlq_workspace_bytes.argtypes = [C.c_int64, C.c_int64, C.c_int64, C.c_int, C.c_int, C.c_int]
    L.bcjr_ldlq_workspace_bytes.restype = C.c_size_t
    L.bcjr_ldlq_viterbi.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_void_p, C.c_int, C.c_int,
                                    C.c_int, C.c_void_p, C.c_int64, C.c_double, C.c_void_p, C.c_void_p,
                                    C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    # block LDL workspace: A (d^2 doubles), the block inverses (d x block doubles), a scalar
    d, b = 512, 64
    assert L.bcjr_block_ldl_workspace_bytes(d, b) >= d * d * 8 + d * b * 8
    assert L.bcjr_block_ldl_workspace_bytes(d, 48) == 0           # d not a multiple of block
    assert L.bcjr_block_ldl_workspace_bytes(0, 1) == 0
    bl = L.bcjr_block_ldl
    assert bl(FAKE, d, 48, 0.0, FAKE, None, FAKE, 1 << 30, None) == -1
    assert bl(FAKE, d, b, -0.1, FAKE, None, FAKE, 1 << 30, None) == -1
    assert bl(None, d, b, 0.0, FAKE, None, FAKE, 1 << 30, None) == -1
    assert bl(FAKE, d, b, 0.0, FAKE + 4, None, FAKE, 1 << 30, None) == -1   # M not 8-byte aligned
    assert bl(FAKE, d, b, 0.0, FAKE, None, None, 0, None) == -3
    assert bl(FAKE, d, b, 0.0, FAKE, None, FAKE, 1024, None) == -3
    ws = L.bcjr_ldlq_workspace_bytes
    assert ws(16, 512, 256, 16, 2, 1) > 512 * 512 * 8
    assert ws(16, 512, 256, 16, 4, 2) > 0
    assert ws(16, 512, 255, 16, 2, 1) == 0
    assert ws(16, 512, 256, 16, 2, 3) == 0                        # V = 3 has no decode
    lv = L.bcjr_ldlq_viterbi
    args = [FAKE, 16, 512, FAKE, 16, 2, 1, FAKE, 256, 0.01, FAKE, FAKE, None, FAKE, 1 << 40, None]
    bad = list(args); bad[8] = 255
    assert lv(*bad) == -1
    bad = list(args); bad[10] = None
    assert lv(*bad) == -1
    bad = list(args); bad[3] = MISALIGNED
    assert lv(*bad) == -1
    bad = list(args); bad[13] = None; bad[14] = 0
    assert lv(*bad) == -3
    bad = list(args); bad[14] = 1024
    assert lv(*bad) == -3

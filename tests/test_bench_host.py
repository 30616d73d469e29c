"""bench.py's host-side contract: one GPU only, the roofline model the JSON
line is priced against, and the measured-traffic table's keys."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (module level imports no GPU library)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_alu_roofline_of_the_scalar_kernel():
    # 16 edges per K x K group-step at K = 4; 97 VALU at the published 128
    # fp32 lanes per clock per CU (157.3 TFLOP/s) and 11 transcendentals at
    # R_T; 256 CUs at 2.4 GHz.  At R_T = 16 this is 6.80e12 edges/s, at 32
    # 8.92e12; at 64 lanes and R_T = 32 (round one's model) 5.287e12.
    assert abs(bench.VALU_LANES_PUBLISHED * 2 * 256 * 2.4e9 - 157.3e12) <= 1e-3 * 157.3e12
    for r_t, want in ((16.0, 6.80e12), (32.0, 8.92e12)):
        got = bench.roofline_edges_per_s(r_t)
        t_group = 97.0 / 128 + 11.0 / r_t
        assert abs(got - 16 * 256 * 2.4e9 / t_group) <= 1e-9 * got
        assert abs(got - want) <= 2e-3 * want
    np_ = bench.roofline_edges_per_s(32.0, 64.0)
    assert abs(np_ - 5.287e12) <= 1e-3 * 5.287e12
    # the dCodebook variant adds 6K = 24 VALU per group-step
    dc = bench.roofline_edges_per_s(16.0, dc=True)
    assert abs(dc - 16 * 256 * 2.4e9 / (121.0 / 128 + 11.0 / 16)) <= 1e-9 * dc


def test_alu_roofline_of_the_vector_kernel():
    t_state = (25.0 + 21.0 / 16) / 128 + (2.0 + 5.0 / 16) / 32
    want = 16 * 256 * 2.4e9 / t_state
    assert abs(bench.roofline_vec_edges_per_s(32.0) - want) <= 1e-9 * want


def test_measured_traffic_is_keyed_by_path_and_source_digest():
    assert bench.MEASURED_TRAFFIC
    for (path, digest), value in bench.MEASURED_TRAFFIC.items():
        assert path in ("fwd_vjp", "vec")
        assert len(digest) == 16 and int(digest, 16) >= 0
        assert value > 0
    d = bench.kernel_source_digest()
    assert len(d) == 16 and d == bench.kernel_source_digest()


def test_issue_rate_probe_library_exports_and_rejects_bad_arguments():
    """The probe library the roofline is priced with: its three entry points
    exist, and bad arguments are refused before any GPU call."""
    import ctypes
    import os
    path = os.path.join(bench.ROOT, "paper_2605_10655_amd", "libissue_rates.so")
    if not os.path.exists(path):
        import pytest
        pytest.skip("libissue_rates.so not built")
    lib = ctypes.CDLL(path)
    for name in ("issue_rate_run", "issue_rate_chains", "issue_rate_ops_per_step"):
        assert hasattr(lib, name)
    ms, a, b = ctypes.c_float(), ctypes.c_double(), ctypes.c_double()
    lib.issue_rate_chains.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_double)]
    assert lib.issue_rate_chains(0, 3, 16, 256, ctypes.byref(ms), ctypes.byref(a), ctypes.byref(b)) == -1
    assert lib.issue_rate_chains(2, 8, 16, 256, ctypes.byref(ms), ctypes.byref(a), ctypes.byref(b)) == -1
    assert lib.issue_rate_chains(0, 8, 0, 256, ctypes.byref(ms), ctypes.byref(a), ctypes.byref(b)) == -1
    lib.issue_rate_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_float),
                                   ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    assert lib.issue_rate_run(10, 16, 256, ctypes.byref(ms), ctypes.byref(a), ctypes.byref(b)) == -1
    v, t = ctypes.c_double(), ctypes.c_double()
    lib.issue_rate_ops_per_step.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_double)]
    assert lib.issue_rate_ops_per_step(5, ctypes.byref(v), ctypes.byref(t)) == 0
    assert (v.value, t.value) == (1.0, 1.0)

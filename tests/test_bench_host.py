"""bench.py's host-side contract: one GPU only, the roofline constants the
JSON line is priced against, and the measured-traffic table's keys."""
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
    # 16 edges per K x K group-step at K = 4; 97 VALU at 64 lanes/clk and 11
    # transcendentals at 32 lanes/clk per CU; 256 CUs at 2.4 GHz
    t_group = 97.0 / 64 + 11.0 / 32
    want = 16 * 256 * 2.4e9 / t_group
    assert abs(bench.roofline_edges_per_s() - want) <= 1e-9 * want
    assert abs(want - 5.287e12) <= 1e-3 * 5.287e12


def test_alu_roofline_of_the_vector_kernel():
    t_state = (25.0 + 21.0 / 16) / 64 + (2.0 + 5.0 / 16) / 32
    want = 16 * 256 * 2.4e9 / t_state
    assert abs(bench.roofline_vec_edges_per_s() - want) <= 1e-9 * want
    assert abs(want - 2.034e13) <= 1e-3 * 2.034e13


def test_measured_traffic_is_keyed_by_path_and_source_digest():
    assert bench.MEASURED_TRAFFIC
    for (path, digest), value in bench.MEASURED_TRAFFIC.items():
        assert path in ("fwd_vjp", "vec")
        assert len(digest) == 16 and int(digest, 16) >= 0
        assert value > 0
    d = bench.kernel_source_digest()
    assert len(d) == 16 and d == bench.kernel_source_digest()

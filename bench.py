#!/usr/bin/env python3
"""Benchmark: trellis edge-updates/s of the fused BCJR soft codeword + VJP.

Workload: S = 65536 states (16 state bits), k = 2, L = 256, a 2048 x 2048
unit-variance Gaussian weight matrix (the q/o-projection shape of a
Llama-3.2-1B layer) = 16384 blocks, random N(0,1) codebook, T = 0.05, one
call computing w_soft, logZ and dW (bcjr_soft_codeword_fwd_vjp).  Inputs are
seeded synthetic data resident in HBM before timing starts.

A step is one such call over the whole matrix.  Edges per step are
B * L * S * 2^k.  Prints one JSON line.

--path vec times the paper's own trellis shape on the same matrix: V = 2
weights and 4 bits per step (16 predecessors per state, 128 steps per
256-weight block), a [65536, 2] N(0,1) codebook, fused w_soft + logZ + dW
(bcjr_vec_soft_codeword_fwd_vjp); edges per step B * (L/2) * S * 16.

--op soft | dc | viterbi times another call on the same data (the soft
codeword alone, the fused call with dCodebook, the Viterbi decode); those
lines carry no roofline.

--path anneal times the annealed QAT loop (computed Gaussian codebook, 8 steps
of forward + VJP with dW and dCodebook + Adam, Viterbi snap) on the
2048 x 8192 gate/up-projection shape; one run of the loop, no roofline.

--path anneal_calls times the annealed gate/up-projection workload as library
calls: 8 fused forward + VJP calls with dW and dCodebook on the 2048 x 8192
matrix at temperatures 0.1 -> 0.001, then the Viterbi decode the last call's
soft codeword is checked against; no roofline.

--path ldlq times BlockLDLQ Viterbi rounding (the Hessian-weighted PTQ
reference) of the 2048 x 2048 matrix under a proxy Hessian; no roofline.

--path ste times the BCJR-STE training step on the same matrix instead: the
hard Viterbi forward (viterbi_decode) followed by its backward pass
(bcjr_ste_vjp, dW only); the roofline then covers the VJP launch.  --T
overrides the temperature (below 0.04 the VJP runs its double-float variant,
whose roofline is not the one reported here).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# ALU roofline of the fused kernel: edge-updates/s at full issue of the
# algorithmic VALU and transcendental work of a K x K group-step,
#   t_group = N_V / R_V + N_T / R_T   clocks per CU (issue serialised),
# at 256 CUs and 2.4 GHz.  R_V is the published fp32 vector peak, 157.3
# TFLOP/s = 128 FMA lanes per clock per CU.  R_T, the v_exp/v_log/v_rcp
# rate, has no published figure: the issue-rate probe (--path rates)
# measures it live, as lane-operations per second over 256 CUs at the
# shader clock the probe reads during its own run.  The probe also shows
# that the two kinds of instruction do not overlap (a 1:1 interleave takes
# the sum of their times), which is the serialised form above.  A second
# model prices the same counts at the probe's measured rates for both.
CUS, CLOCK_HZ = 256, 2.4e9
VALU_LANES_PUBLISHED = 128.0     # per CU and clock: 157.3e12 FLOP/s / (2 FLOP x 256 CUs x 2.4e9)
# algorithmic work per K x K group-step, K = 4, fwd + w_soft + logZ + dW
ALG_VALU_PER_GROUP = 97.0
ALG_TRANS_PER_GROUP = 11.0
ALG_DC_VALU_PER_GROUP = 24.0     # + dCodebook: 6K more VALU, no transcendental
EDGES_PER_GROUP = 16.0           # K^2
# vector-emission trellis (K = 16, V = 2): algorithmic work per state-step,
# fwd + w_soft + logZ + dW (backward row: 10 VALU + 1 exp per state, 4 VALU and
# a log and a reciprocal per row; forward column: 15 VALU + 1 exp per state,
# 17 VALU and a log, an exp and a reciprocal per column of 16 states)
ALG_VEC_VALU_PER_STATE = 25.0 + (4.0 + 17.0) / 16.0
ALG_VEC_TRANS_PER_STATE = 2.0 + 5.0 / 16.0
EDGES_PER_STATE_VEC = 16.0

# issue-rate probe operations (csrc/issue_rates.hip)
PROBE_OPS = {"fma_f32": 0, "exp_f32": 1, "log_f32": 2, "rcp_f32": 3, "fma_f64": 4,
             "fma_exp_1to1": 5, "fma_exp_4to1": 6, "fma_exp_8to1": 7, "add_f32": 8, "max_f32": 9}


def issue_rates(iters=16384, grid=4096, ops=None):
    """Runs every probe once (timed with HIP events) and returns per-op
    lane-operations per clock per CU at the shader clock the probe read,
    R_T (the slowest of v_exp, v_log, v_rcp) and R_V_measured (v_fma_f32).
    The default grid, 4096 workgroups of 4 waves, is the occupancy at which
    the probe measured the highest rates (1 to 16 waves per SIMD swept by
    --path rates)."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2605_10655_amd", "libissue_rates.so"))
    lib.issue_rate_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                   ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_double)]
    lib.issue_rate_run.restype = ctypes.c_int
    out = {}
    for name, op in PROBE_OPS.items():
        if ops is not None and name not in ops:
            continue
        ms, cnt, clk = ctypes.c_float(), ctypes.c_double(), ctypes.c_double()
        rc = lib.issue_rate_run(op, iters, grid, ctypes.byref(ms), ctypes.byref(cnt), ctypes.byref(clk))
        if rc != 0:
            raise RuntimeError(f"issue-rate probe {name} failed ({rc})")
        sec = ms.value / 1e3
        out[name] = {"ms": ms.value, "lane_ops": cnt.value, "clock_ghz": clk.value / 1e9,
                     "lanes_per_clk_cu": cnt.value / (sec * CUS * clk.value),
                     "lane_ops_per_s": cnt.value / sec}
    if ops is not None:
        return {"ops": out}
    fma = out["fma_f32"]["lane_ops_per_s"]
    r_t = min(out[k]["lanes_per_clk_cu"] for k in ("exp_f32", "log_f32", "rcp_f32"))
    # serialised issue predicts a 1:1 interleave at 1/(1/fma + 1/trans) per pair
    exp = out["exp_f32"]["lane_ops_per_s"]
    pair_s = out["fma_exp_1to1"]["ms"] / 1e3
    pairs = out["fma_exp_1to1"]["lane_ops"] / 2
    serial_s = pairs / fma + pairs / exp
    overlap_s = max(pairs / fma, pairs / exp)
    return {"ops": out, "R_T": r_t, "R_V_measured": out["fma_f32"]["lanes_per_clk_cu"],
            "fma_exp_1to1_s": pair_s, "serialised_model_s": serial_s,
            "overlapped_model_s": overlap_s}


def chain_intervals(iters=4096):
    """Mean shader cycles per VALU instruction of one wave with 2, 4, 8, 16 and
    32 independent chains per lane, for v_fma_f32 and v_add_f32, at 1, 2 and 4
    waves per SIMD: {op: {waves_per_simd: {chains: cycles}}}."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2605_10655_amd", "libissue_rates.so"))
    lib.issue_rate_chains.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_double)]
    lib.issue_rate_chains.restype = ctypes.c_int
    out = {}
    for op, name in ((0, "fma_f32"), (1, "add_f32")):
        out[name] = {}
        for wps in (1, 2, 4):
            row = {}
            for chains in (2, 4, 8, 16, 32):
                ms, cyc, clk = ctypes.c_float(), ctypes.c_double(), ctypes.c_double()
                rc = lib.issue_rate_chains(op, chains, iters, 256 * wps, ctypes.byref(ms),
                                           ctypes.byref(cyc), ctypes.byref(clk))
                if rc != 0:
                    raise RuntimeError(f"chain probe {name}/{chains} failed ({rc})")
                row[chains] = round(cyc.value, 2)
            out[name][wps] = row
    return out


def roofline_edges_per_s(r_t, r_v=VALU_LANES_PUBLISHED, dc=False) -> float:
    n_v = ALG_VALU_PER_GROUP + (ALG_DC_VALU_PER_GROUP if dc else 0.0)
    t_group = n_v / r_v + ALG_TRANS_PER_GROUP / r_t
    return EDGES_PER_GROUP * CUS * CLOCK_HZ / t_group


def roofline_vec_edges_per_s(r_t, r_v=VALU_LANES_PUBLISHED) -> float:
    t_state = ALG_VEC_VALU_PER_STATE / r_v + ALG_VEC_TRANS_PER_STATE / r_t
    return EDGES_PER_STATE_VEC * CUS * CLOCK_HZ / t_state


# HBM bytes per launch of the timed kernel, from two rocprofv3 --pmc passes
# (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0: the factors that map a plain 1 GiB
# device copy's readings to its 1 GiB read and written), keyed by a digest of
# the sources that define that kernel (its headers, translation unit and
# build flags, and the argument block).
# Any other source reports null.
MEASURED_TRAFFIC = {
    ("fwd_vjp", "6f9f29842f82571d"): 2.68507e8 * 1024 * 2.0 + 5.36960e8 * 1024 * 1.0,
}
KERNEL_SOURCES = {"fwd_vjp": ("bcjr_rot_kernels.h", "bcjr_rot.hip", "bcjr_device.h", "bcjr_internal.h",
                              "../build.py"),
                  "vec": ("bcjr_vec_kernels.h", "bcjr_kernels.h", "bcjr_device.h", "bcjr_internal.h"),
                  # the log-domain and double-float kernels (dCodebook, T < 0.04) and their dispatcher
                  "log": ("bcjr_kernels.h", "bcjr_device.h", "bcjr_internal.h", "bcjr_capi.hip"),
                  # the pruned low-temperature VJP (with its double-float repair pass)
                  "pruned": ("bcjr_pruned_kernels.h", "bcjr_kernels.h", "bcjr_device.h", "bcjr_internal.h",
                             "bcjr_capi.hip")}


def kernel_source_digest(path: str = "fwd_vjp") -> str:
    """SHA-256 (16 hex) of a path's kernel sources with comments and blank space removed."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[path]:
        with open(os.path.join(ROOT, "paper_2605_10655_amd", "csrc", name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(target_s: float = 15.0):
    """The fp64 oracle on a bounded sample of the same workload (host cores)."""
    import numpy as np
    from oracle import oracle as O
    from paper_2605_10655_amd import workloads as WL
    wl = WL.workload(4)
    cores = O.default_threads()
    c = WL.codebook(4)
    w = WL.weights(4, rows=32)                      # 256 blocks available
    g = WL.upstream(4, B=w.shape[0])
    T = float(np.float32(wl.temps[0]))
    # calibrate with one block per core, then scale to ~target_s
    nb = min(cores, w.shape[0])
    t0 = time.time()
    O.soft_codeword_vjp(w[:nb], c, wl.state_bits, wl.k, T, g[:nb], want_dc=False, nthreads=cores)
    t1 = time.time() - t0
    rounds = max(1, min(int(target_s / max(t1, 1e-3)), w.shape[0] // nb))
    if rounds > 1:
        nb2 = nb * rounds
        t0 = time.time()
        O.soft_codeword_vjp(w[:nb2], c, wl.state_bits, wl.k, T, g[:nb2], want_dc=False,
                            nthreads=cores)
        nb, t1 = nb2, time.time() - t0
    edges = nb * wl.L * wl.S * (1 << wl.k)
    return {"value": edges / t1, "unit": "edge-updates/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{nb} blocks of the same matrix (first rows), fwd+logZ+dW, fp64, {t1:.1f} s"}


def run_anneal(args):
    """The annealing loop on the gate/up-projection shape: 2048 x 8192 N(0,1)
    weights as 65536 blocks of 256, S = 65536, k = 2, computed Gaussian
    codebook, the layer-output loss tr(R H R^T) with a proxy Hessian of
    synthetic inputs, 8 steps T = 0.1 -> 0.001, each a forward call and a VJP
    call (dW and dCodebook) with Adam on the weights and the codebook, then
    the Viterbi snap (losses per weight reported against the snap of the
    initial weights).  Edges are counted as B * L * S * K per step (one forward +
    VJP unit, as in the headline metric)."""
    import numpy as np
    import torch
    import paper_2605_10655_amd as P
    from paper_2605_10655_amd import workloads as WL
    from paper_2605_10655_amd.qat import QATConfig, anneal_qat
    wl = WL.workload(5)
    dev = torch.device("cuda:0")
    rows, cols = wl.rows, wl.cols
    W0 = torch.from_numpy(WL.weights(5)).to(dev).view(rows, cols)
    c = P.bcjr_gaussian_codebook(wl.state_bits, 1, seed=5)
    # proxy Hessian of the layer-output error from synthetic calibration inputs
    X = torch.from_numpy(WL.calibration_inputs(5)).to(dev)
    H = (X.T @ X) / X.shape[0]
    del X
    cfg = QATConfig(state_bits=wl.state_bits, k=wl.k, block=wl.L, T0=0.1, T_end=1e-3, steps=8,
                    lr=1e-3, grad_clip=1.0, learn_codebook=True, lr_codebook=1e-4)
    if args.warmup:
        small = QATConfig(**{**cfg.__dict__, "steps": 2})
        anneal_qat(W0[:8], c, small, H=H)
        torch.cuda.synchronize()
        print("warmup done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    res = anneal_qat(W0, c, cfg, H=H)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    B = rows * cols // wl.L
    edges = cfg.steps * B * wl.L * wl.S * (1 << wl.k)
    rec = {
        "metric": "annealed QAT loop: trellis edge-updates/s over 8 fwd+VJP(dW, dCodebook)+Adam steps "
                  "and the Viterbi snap, S=65536, k=2, L=256",
        "value": edges / wall, "unit": "edge-updates/s", "n_gpus": 1, "steps": cfg.steps,
        "warmup": args.warmup, "ms_per_step": wall * 1e3 / cfg.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "2048x8192 N(0,1) weights as 65536 blocks of L=256; S=65536, k=2, "
                               "computed Gaussian codebook; layer-output loss with a proxy Hessian "
                               "H = X^T X / 4096 of synthetic inputs; T 0.1 -> 0.001 in 8 steps; "
                               "Adam on W (lr 1e-3, clip 1) and the codebook (lr 1e-4)",
                   "B": B, "L": wl.L, "S": wl.S, "k": wl.k, "temps": res.temps},
        "seconds": wall, "roofline": None,
        "loss_per_step": [l / W0.numel() for l in res.losses],
        "loss_hard": res.loss_hard / W0.numel(), "loss_ptq": res.loss_ptq / W0.numel(),
        "max_drift": res.max_drift, "drift_budget": res.budget,
    }
    print(json.dumps(rec), flush=True)


def anneal_calls_record(warmup, r_t):
    """The annealed gate/up-projection workload as a sequence of library
    calls: 2048 x 8192 N(0,1) weights as 65536 blocks of 256, S = 65536,
    k = 2, N(0,1) codebook, 8 successive calls of the fused forward + VJP
    with dW and dCodebook at T_i = 0.1 (0.01)^(i/7) (a fresh upstream
    gradient per call; the precision switch puts the last six on the
    double-float kernel), then the Viterbi decode of the same blocks, against
    which the last call's soft codeword is checked (the fraction of weights
    whose soft codeword sits within 2e-5 of the minimum-distortion codeword).
    A step is one call; edges per call are B * L * S * K.  The roofline is
    the fwd + dW + dCodebook model (121 VALU + 11 transcendentals per
    group-step)."""
    import torch
    import paper_2605_10655_amd as P
    from paper_2605_10655_amd import workloads as WL
    wl = WL.workload(5)
    dev = torch.device("cuda:0")
    n, k, L = wl.state_bits, wl.k, wl.L
    w = torch.from_numpy(WL.weights(5)).to(dev)
    c = torch.from_numpy(WL.codebook(5)).to(dev)
    B = w.shape[0]
    w_soft = torch.empty_like(w)
    logZ = torch.empty(B, dtype=torch.float32, device=dev)
    dW = torch.empty_like(w)
    dc = torch.empty_like(c)
    ws = torch.empty(P.bcjr_workspace_bytes(B, L, n, k, P.OP_FWD_VJP), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    temps = [float(T) for T in wl.temps]
    gs = [torch.from_numpy(WL.upstream(5, i)).to(dev) for i in range(len(temps))]

    def call(T, g):
        P.bcjr_soft_codeword_fwd_vjp(w, c, n, k, T, g, w_soft=w_soft, logZ=logZ, dW=dW,
                                     dCodebook=dc, workspace=ws, stream=stream)

    for _ in range(warmup):  # one call on each kernel (fp32 and double-float)
        call(temps[0], gs[0])
        call(temps[-1], gs[-1])
        torch.cuda.synchronize()
        print("anneal calls: warmup done", file=sys.stderr, flush=True)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in temps]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for (a, b), T, g in zip(ev, temps, gs):
        a.record(stream)
        call(T, g)
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = [a.elapsed_time(b) for a, b in ev]
    print("anneal calls: per call ms " + " ".join(f"{x:.0f}" for x in call_ms), file=sys.stderr,
          flush=True)
    _, w_hard = P.viterbi_decode(w, c, n, k)
    torch.cuda.synchronize()
    agree = float(((w_soft - w_hard).abs() <= 2e-5).float().mean().item())
    edges = len(temps) * B * L * wl.S * (1 << k)
    peak = roofline_edges_per_s(r_t, dc=True)
    del ws
    torch.cuda.empty_cache()
    return {
        "value": edges / wall, "unit": "edge-updates/s", "seconds": wall, "call_ms": call_ms,
        "temps": temps, "B": B, "roofline_peak": peak, "roofline_frac": edges / wall / peak,
        "final_call_soft_equals_viterbi_frac": agree,
    }


def run_anneal_calls(args):
    import torch
    rates = issue_rates()
    r = anneal_calls_record(args.warmup, rates["R_T"])
    rec = {
        "metric": "trellis edge-updates/s fwd+VJP incl. dCodebook, 8 annealed calls at S=65536,k=2,L=256",
        "value": r["value"], "unit": "edge-updates/s", "n_gpus": 1, "steps": 8,
        "warmup": args.warmup, "ms_per_step": r["seconds"] * 1e3 / 8, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 (double-float log vectors below T=0.04)",
        "data": "synthetic",
        "config": {"workload": "2048x8192 N(0,1) weights as 65536 blocks of L=256; S=65536, k=2, "
                               "N(0,1) codebook; 8 calls of fused w_soft+logZ+dW+dCodebook, "
                               "T 0.1 -> 0.001 geometric, fresh upstream gradient per call",
                   "B": r["B"], "L": 256, "S": 65536, "k": 2, "temps": r["temps"]},
        "seconds": r["seconds"], "call_ms": r["call_ms"],
        "roofline": {"bound": "alu", "achieved": r["value"] / 1e9, "peak": r["roofline_peak"] / 1e9,
                     "unit": "Gedge/s", "frac": r["roofline_frac"], "traffic": None,
                     "model": "121 VALU / 128 lanes + 11 trans / R_T per 16-edge group-step",
                     "R_T": rates["R_T"]},
        "final_call_soft_equals_viterbi_frac": r["final_call_soft_equals_viterbi_frac"],
    }
    print(json.dumps(rec), flush=True)


def run_config(args):
    """Configs 1-3, full batch: one step is the fused call at every listed
    temperature (w_soft + logZ + dW, with dCodebook for configs 1 and 3,
    and for config 1 the Viterbi decode too).  Edges per step are the sum
    over the temperatures of B * L * S * K.  The oracle is timed on the same
    step (fp64, all host cores): every block when that takes under about
    30 s, else the first blocks it covers in that time."""
    import numpy as np
    import torch
    import paper_2605_10655_amd as P
    from paper_2605_10655_amd import workloads as WL
    from oracle import oracle as O
    cfg = args.config
    wl = WL.workload(cfg)
    torch.zeros(1, device="cuda:0")
    rates = issue_rates()
    r_t = rates["R_T"]
    want_dc = "dc" in wl.outputs
    want_vit = "viterbi" in wl.outputs
    n, k, L = wl.state_bits, wl.k, wl.L
    dev = torch.device("cuda:0")
    cw, ww, gw = WL.codebook(cfg), WL.weights(cfg), WL.upstream(cfg)
    w, c, g = (torch.from_numpy(a).to(dev) for a in (ww, cw, gw))
    B = w.shape[0]
    w_soft, dW = torch.empty_like(w), torch.empty_like(w)
    logZ = torch.empty(B, dtype=torch.float32, device=dev)
    dc = torch.empty_like(c) if want_dc else None
    states = torch.empty((B, L), dtype=torch.int32, device=dev)
    w_hard = torch.empty_like(w)
    ws = torch.empty(max(P.bcjr_workspace_bytes(B, L, n, k, P.OP_FWD_VJP),
                         P.bcjr_workspace_bytes(B, L, n, k, P.OP_VITERBI)),
                     dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    temps = [float(T) for T in wl.temps]

    def step():
        for T in temps:
            P.bcjr_soft_codeword_fwd_vjp(w, c, n, k, T, g, w_soft=w_soft, logZ=logZ, dW=dW,
                                         dCodebook=dc, want_dCodebook=want_dc, workspace=ws,
                                         stream=stream)
        if want_vit:
            P.viterbi_decode(w, c, n, k, states=states, w_hard=w_hard, workspace=ws, stream=stream)

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    a.record(stream)
    for _ in range(args.steps):
        step()
    b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_s = a.elapsed_time(b) / 1e3 / args.steps
    edges = len(temps) * wl.edges
    peak = roofline_edges_per_s(r_t, dc=want_dc)
    print(f"config {cfg}: {wall * 1e3 / args.steps:.3f} ms/step; timing the oracle ...",
          file=sys.stderr, flush=True)

    def oracle_on(lo, hi):
        for T in temps:
            O.soft_codeword_vjp(ww[lo:hi], cw, n, k, float(np.float32(T)), gw[lo:hi], want_dc=want_dc)
        if want_vit:
            O.viterbi(ww[lo:hi], cw, n, k)

    # every block when the oracle needs under ~30 s for them, else the first
    # blocks it covers in that time (timed in chunks, progress on stderr)
    probe = min(B, 64)
    t0 = time.perf_counter()
    oracle_on(0, probe)
    cpu_s = time.perf_counter() - t0
    nb = B if cpu_s * B / probe <= 30.0 else min(B, max(probe, int(probe * 30.0 / cpu_s)))
    done = probe
    while done < nb:
        hi = min(nb, done + 1024)
        t0 = time.perf_counter()
        oracle_on(done, hi)
        cpu_s += time.perf_counter() - t0
        done = hi
        print(f"oracle: {done} of {nb} blocks, {cpu_s:.1f} s", file=sys.stderr, flush=True)
    cpu_edges = edges * nb / B
    rec = {
        "metric": f"trellis edge-updates/s fwd+VJP, config {cfg} ({wl.name})",
        "value": edges / (wall / args.steps), "unit": "edge-updates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name + "; fused " + "+".join(
            o for o in wl.outputs if o != "viterbi") + (" + Viterbi" if want_vit else "") +
            f" at T in {temps}, full batch", "B": B, "L": L, "S": wl.S, "k": k, "temps": temps},
        "blocks_per_s": B * len(temps) / (wall / args.steps),
        "roofline": {"bound": "alu", "achieved": edges / kern_s / 1e9, "peak": peak / 1e9,
                     "unit": "Gedge/s", "frac": edges / kern_s / peak, "traffic": None,
                     "kernel_ms": kern_s * 1e3, "R_T": r_t},
        "cpu_baseline": {"value": cpu_edges / cpu_s, "unit": "edge-updates/s",
                         "cores": O.default_threads(), "kind": "oracle", "cpu": cpu_model(),
                         "sample": (f"all {B} blocks" if nb == B else f"the first {nb} of {B} blocks")
                         + f", every temperature, {cpu_s:.1f} s"},
    }
    print(json.dumps(rec), flush=True)


def run_rates(args):
    """The gfx950 issue-rate probe alone: one JSON line of lane-operations
    per clock per CU for each probed instruction, the clock the probe read,
    R_T, and the 1:1 fma + exp interleave against the serialised and
    overlapped issue models.  Then one line per occupancy: grids of 256 to
    4096 workgroups of 4 waves are 1 to 16 waves per SIMD."""
    import torch
    torch.zeros(1, device="cuda:0")
    for grid in (256, 512, 1024, 2048, 4096):
        r = issue_rates(grid=grid, ops=("fma_f32", "add_f32", "exp_f32", "fma_f64", "fma_exp_1to1"))
        print(json.dumps({"grid": grid, "waves_per_simd": grid // 256,
                          "lanes_per_clk_cu": {k: round(v["lanes_per_clk_cu"], 2)
                                               for k, v in r["ops"].items()},
                          "clock_ghz": {k: round(v["clock_ghz"], 3) for k, v in r["ops"].items()}}),
              flush=True)
    r = issue_rates()
    ops = {k: {kk: v[kk] for kk in ("ms", "lanes_per_clk_cu", "clock_ghz", "lane_ops")}
           for k, v in r["ops"].items()}
    rec = {"metric": "gfx950 VALU issue rates (lane-ops per clock per CU)", "ops": ops,
           "R_T": r["R_T"], "R_V_measured": r["R_V_measured"],
           "fma_exp_1to1_s": r["fma_exp_1to1_s"],
           "serialised_model_s": r["serialised_model_s"],
           "overlapped_model_s": r["overlapped_model_s"],
           "probe": "csrc/issue_rates.hip: 4096 workgroups x 256 lanes, 16384 steps of 8 "
                    "independent chains per lane"}
    print(json.dumps(rec), flush=True)
    # dependency latency: shader cycles per VALU instruction of one wave for
    # 2..32 independent chains per lane at 1, 2 and 4 waves per SIMD
    lat = chain_intervals()
    print(json.dumps({"metric": "gfx950 cycles per VALU instruction per wave, by independent "
                                "chains per lane (v_fma_f32 VOP3 / v_add_f32 VOP2)",
                      "cycles_per_instr": lat,
                      "probe": "csrc/issue_rates.hip chain_kernel: 256 x waves-per-SIMD "
                               "workgroups of 256 lanes, 4096 x 4 steps per chain"}), flush=True)


def run_ldlq(args):
    """BlockLDLQ Viterbi rounding of the 2048 x 2048 N(0,1) matrix (S = 65536,
    k = 2, blocks of 256 columns) under the proxy Hessian of synthetic
    inputs: 8 column blocks, each one batched Viterbi call over the 2048 rows
    plus the feedback GEMM.  Reports the time of the whole rounding and the
    Hessian-weighted loss against the plain per-block Viterbi codeword."""
    import numpy as np
    import torch
    import paper_2605_10655_amd as P
    from paper_2605_10655_amd import workloads as WL
    from paper_2605_10655_amd.ldlq import hw_loss, ldlq_viterbi
    wl = WL.workload(4)
    dev = torch.device("cuda:0")
    rows, cols = wl.rows, wl.cols
    W = torch.from_numpy(WL.weights(4)).to(dev).view(rows, cols)
    c = torch.from_numpy(WL.codebook(4)).to(dev)
    X = torch.from_numpy(WL.calibration_inputs(4)).to(dev)
    H = (X.T @ X) / X.shape[0]
    del X
    for _ in range(args.warmup):
        ldlq_viterbi(W, c, wl.state_bits, wl.k, H, block=wl.L)
        torch.cuda.synchronize()
    times = []
    for _ in range(max(1, args.steps)):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        Wh, _ = ldlq_viterbi(W, c, wl.state_bits, wl.k, H, block=wl.L)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    _, plain = P.viterbi_decode(W.reshape(-1, wl.L), c, wl.state_bits, wl.k)
    torch.cuda.synchronize()
    sec = float(np.median(times))
    B = rows * cols // wl.L
    rec = {
        "metric": "BlockLDLQ Viterbi rounding: trellis edge-updates/s (Viterbi) at S=65536,k=2,L=256",
        "value": B * wl.L * wl.S * (1 << wl.k) / sec, "unit": "edge-updates/s", "n_gpus": 1,
        "steps": len(times), "warmup": args.warmup, "ms_per_step": sec * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64 metrics",
        "data": "synthetic",
        "config": {"workload": "2048x2048 N(0,1) weights, S=65536, k=2, blocks of 256 columns; "
                               "proxy Hessian H = X^T X / 4096 of synthetic inputs, damp 0.01",
                   "B": B, "L": wl.L, "S": wl.S, "k": wl.k},
        "roofline": None,
        "hw_loss_ldlq": hw_loss(W, Wh, H) / W.numel(),
        "hw_loss_plain_viterbi": hw_loss(W, plain.view(rows, cols), H) / W.numel(),
    }
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--path", choices=("fwd_vjp", "ste", "vec", "anneal", "anneal_calls", "ldlq",
                                       "rates"), default="fwd_vjp")
    ap.add_argument("--config", type=int, choices=(1, 2, 3, 4, 5), default=4,
                    help="workload: 4 (default) is the headline S=65536 q/o-projection call; 1-3 "
                         "the small and mid trellises (full batch, every listed temperature, "
                         "oracle timed on every block); 5 the 8 annealed gate/up-projection calls")
    ap.add_argument("--no-extras", action="store_true",
                    help="headline line only: skip the separate-call and 8-call annealed timings")
    ap.add_argument("--T", type=float, default=None)
    ap.add_argument("--op", choices=("fwd_vjp", "soft", "dc", "viterbi"), default="fwd_vjp",
                    help="call timed on the fwd_vjp and vec paths: the fused w_soft+logZ+dW call "
                         "(default), the soft codeword + logZ alone, w_soft+logZ+dW+dCodebook, or "
                         "the Viterbi decode; only the default carries a roofline")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device-to-device copy of this many bytes (the "
                         "reference kernel for scaling FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(blocks are independent: N GPUs would each run B/N blocks)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2605_10655_amd as P
    from paper_2605_10655_amd import workloads as WL

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.copy_bytes:
        src = torch.empty(args.copy_bytes // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        # then the copy's own rate (bytes read + written), HIP events, 5 copies
        st = torch.cuda.current_stream()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(st)
        for _ in range(5):
            dst.copy_(src)
        t1.record(st)
        torch.cuda.synchronize()
        sec = t0.elapsed_time(t1) / 1e3 / 5
        print(json.dumps({"copy_bytes": src.numel() * 4,
                          "copy_read_plus_write_bytes_per_s": 2 * src.numel() * 4 / sec}), flush=True)
        return
    P.load_library()
    if args.path == "anneal":
        run_anneal(args)
        return
    if args.path == "anneal_calls":
        run_anneal_calls(args)
        return
    if args.path == "ldlq":
        run_ldlq(args)
        return
    if args.path == "rates":
        run_rates(args)
        return
    if args.config == 5:
        run_anneal_calls(args)
        return
    if args.config in (1, 2, 3):
        run_config(args)
        return
    torch.zeros(1, device="cuda:0")
    rates = issue_rates()
    print(f"issue rates (lanes/clk/CU): R_T = {rates['R_T']:.2f}, fma "
          f"{rates['R_V_measured']:.1f} at {rates['ops']['fma_f32']['clock_ghz']:.2f} GHz",
          file=sys.stderr, flush=True)
    wl = WL.workload(4)
    n, k, L, T = wl.state_bits, wl.k, wl.L, wl.temps[0] if args.T is None else args.T
    ste = args.path == "ste"
    vec = args.path == "vec"
    dev = torch.device("cuda:0")
    w = torch.from_numpy(WL.weights(4)).to(dev)
    c = torch.from_numpy(WL.codebook_vec(4) if vec else WL.codebook(4)).to(dev)
    g = torch.from_numpy(WL.upstream(4)).to(dev)
    B = w.shape[0]
    w_soft = torch.empty_like(w)
    logZ = torch.empty(B, dtype=torch.float32, device=dev)
    dW = torch.empty_like(w)
    states = torch.empty((B, L), dtype=torch.int32, device=dev) if ste else None
    if vec:
        k = 4
    ws_bytes = (P.bcjr_vec_workspace_bytes(B, L, n, k, 2, P.OP_FWD_VJP) if vec
                else P.bcjr_workspace_bytes(B, L, n, k, P.OP_FWD_VJP))
    if ste:
        ws_bytes = max(ws_bytes, P.bcjr_workspace_bytes(B, L, n, k, P.OP_VITERBI))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    op = "fwd_vjp" if ste else args.op
    dc_out = torch.empty_like(c) if op == "dc" else None
    vstates = torch.empty((B, L // 2 if vec else L), dtype=torch.int32, device=dev)
    if op == "viterbi":
        ws_bytes = (P.bcjr_vec_workspace_bytes(B, L, n, k, 2, P.OP_VITERBI) if vec
                    else P.bcjr_workspace_bytes(B, L, n, k, P.OP_VITERBI))
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)

    def step(mid=None):
        if op == "soft":
            if vec:
                P.bcjr_vec_soft_codeword(w, c, n, k, 2, T, w_soft=w_soft, logZ=logZ, workspace=ws,
                                         stream=stream)
            else:
                P.bcjr_soft_codeword(w, c, n, k, T, w_soft=w_soft, logZ=logZ, workspace=ws,
                                     stream=stream)
        elif op == "viterbi":
            if vec:
                P.bcjr_vec_viterbi_decode(w, c, n, k, 2, states=vstates, w_hard=w_soft,
                                          workspace=ws, stream=stream)
            else:
                P.viterbi_decode(w, c, n, k, states=vstates, w_hard=w_soft, workspace=ws,
                                 stream=stream)
        elif op == "dc":
            if vec:
                P.bcjr_vec_soft_codeword_fwd_vjp(w, c, n, k, 2, T, g, w_soft=w_soft, logZ=logZ,
                                                 dW=dW, dCodebook=dc_out, workspace=ws,
                                                 stream=stream)
            else:
                P.bcjr_soft_codeword_fwd_vjp(w, c, n, k, T, g, w_soft=w_soft, logZ=logZ, dW=dW,
                                             dCodebook=dc_out, workspace=ws, stream=stream)
        elif ste:
            P.viterbi_decode(w, c, n, k, states=states, w_hard=w_soft, workspace=ws,
                             stream=stream)
            if mid is not None:
                mid.record(stream)
            P.bcjr_ste_vjp(w, c, n, k, T, w_soft, g, dW=dW, want_dCodebook=False, workspace=ws,
                           stream=stream)
        elif vec:
            P.bcjr_vec_soft_codeword_fwd_vjp(w, c, n, k, 2, T, g, w_soft=w_soft, logZ=logZ, dW=dW,
                                             want_dCodebook=False, workspace=ws, stream=stream)
        else:
            P.bcjr_soft_codeword_fwd_vjp(w, c, n, k, T, g, w_soft=w_soft, logZ=logZ, dW=dW,
                                         want_dCodebook=False, workspace=ws, stream=stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print(f"warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)

    # events recorded on the stream the kernels are launched on
    # (the STE step's VJP launch starts at the event recorded after its decode)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(ev[i][2] if ste else None)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kernel_ms = [(m if ste else a).elapsed_time(b) for a, b, m in ev]
    ms_per_step = wall * 1e3 / args.steps
    edges = B * (L // 2) * wl.S * 16 if vec else wl.edges
    value = edges / (ms_per_step / 1e3)
    kern_avg_s = float(np.mean(kernel_ms)) / 1e3
    achieved = edges / kern_avg_s
    r_t = rates["R_T"]
    peak = roofline_vec_edges_per_s(r_t) if vec else roofline_edges_per_s(r_t)
    r_vm = rates["R_V_measured"]
    peak_m = (roofline_vec_edges_per_s(r_t, r_vm) if vec else roofline_edges_per_s(r_t, r_vm))
    print(f"timed {args.steps} steps: {ms_per_step:.1f} ms/step (events avg {kern_avg_s * 1e3:.1f} ms)",
          file=sys.stderr, flush=True)

    op_what = {"fwd_vjp": "fused w_soft+logZ+dW", "soft": "soft codeword + logZ",
               "dc": "fused w_soft+logZ+dW+dCodebook", "viterbi": "Viterbi decode"}[op]
    op_metric = {"fwd_vjp": "fwd+VJP", "soft": "soft codeword", "dc": "fwd+VJP incl. dCodebook",
                 "viterbi": "Viterbi"}[op]
    if vec:
        metric = (f"trellis edge-updates/s {op_metric} at S=65536, 16 predecessors (4 bits/step), "
                  "V=2, 256-weight blocks")
        what = f"V=2, 4 bits per step (128 steps per block), [65536,2] N(0,1) codebook; {op_what}"
    elif ste:
        metric = "trellis edge-updates/s BCJR-STE step (Viterbi fwd + VJP) at S=65536,k=2,L=256"
        what = "BCJR-STE step: viterbi_decode + bcjr_ste_vjp (dW)"
    elif op == "fwd_vjp":
        metric = "trellis edge-updates/s fwd+VJP at S=65536,k=2,L=256; % VALU roofline"
        what = "fused w_soft+logZ+dW"
    else:
        metric = f"trellis edge-updates/s {op_metric} at S=65536,k=2,L=256"
        what = op_what
    rec = {
        "metric": metric,
        "value": value,
        "unit": "edge-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"2048x2048 N(0,1) weights as 16384 blocks of L=256; S=65536, k={k}, "
                               f"T={T}; {what}",
                   "B": B, "L": L, "S": wl.S, "k": k, "V": 2 if vec else 1, "T": T},
        "blocks_per_s": B / (ms_per_step / 1e3),
        "roofline": None if op != "fwd_vjp" else {
            "bound": "alu", "achieved": achieved / 1e9, "peak": peak / 1e9,
            "unit": "Gedge/s", "frac": achieved / peak,
            "traffic": None if (ste or args.T is not None)
            else MEASURED_TRAFFIC.get((args.path, kernel_source_digest(args.path))),
            "kernel_ms": kern_avg_s * 1e3,
            "model": ("per state-step %.2f VALU / R_V + %.4f trans / R_T" %
                      (ALG_VEC_VALU_PER_STATE, ALG_VEC_TRANS_PER_STATE)) if vec else
                     ("per 16-edge group-step %g VALU / R_V + %g trans / R_T at 256 CUs x 2.4 GHz"
                      % (ALG_VALU_PER_GROUP, ALG_TRANS_PER_GROUP)),
            "R_V": VALU_LANES_PUBLISHED, "R_T": r_t,
            "R_V_measured": r_vm, "peak_measured_rates": peak_m / 1e9,
            "frac_measured_rates": achieved / peak_m},
    }
    if op != "fwd_vjp":
        rec["kernel_ms"] = kern_avg_s * 1e3
    headline = not ste and not vec and args.T is None and op == "fwd_vjp"
    if headline and not args.no_extras:
        # the same work as the autograd node issues it: the soft codeword
        # call, then the VJP call (dW), each a forward-backward pass
        sep = []
        for i in range(args.warmup + 3):
            a, m, b = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            a.record(stream)
            P.bcjr_soft_codeword(w, c, n, k, T, w_soft=w_soft, logZ=logZ, workspace=ws, stream=stream)
            m.record(stream)
            P.bcjr_soft_codeword_vjp(w, c, n, k, T, g, dW=dW, want_dCodebook=False, workspace=ws,
                                     stream=stream)
            b.record(stream)
            torch.cuda.synchronize()
            if i >= args.warmup:
                sep.append((a.elapsed_time(m), m.elapsed_time(b)))
        soft_ms = float(np.median([x[0] for x in sep]))
        vjp_ms = float(np.median([x[1] for x in sep]))
        rec["separate_calls"] = {"soft_ms": soft_ms, "vjp_ms": vjp_ms, "total_ms": soft_ms + vjp_ms,
                                 "edges_per_s": edges / ((soft_ms + vjp_ms) / 1e3),
                                 "what": "bcjr_soft_codeword then bcjr_soft_codeword_vjp (dW), "
                                         "median of 3"}
        print(f"separate calls: {soft_ms:.1f} + {vjp_ms:.1f} ms", file=sys.stderr, flush=True)
        del ws
        torch.cuda.empty_cache()
        print("timing the 8 annealed gate/up-projection calls ...", file=sys.stderr, flush=True)
        rec["anneal_calls"] = anneal_calls_record(1, r_t)
    if headline:
        rec["issue_rates"] = {k2: round(v["lanes_per_clk_cu"], 3) for k2, v in rates["ops"].items()}
        rec["issue_rates"]["clock_ghz"] = rates["ops"]["fma_f32"]["clock_ghz"]
    if not args.no_cpu_baseline and headline:
        print("timing the oracle on the host cores ...", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()

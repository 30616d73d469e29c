"""Seeded synthetic inputs for the BCJR soft-codeword workloads.

This module only draws random numbers; it holds none of the method's
arithmetic and is shared by the tests, the benchmark and the CPU oracle
checks.  Draws are float64 from numpy's PCG64 and are cast to float32; both
the GPU path and the oracle receive the same float32 arrays.

Blocks are consecutive runs of L weights in a row-major weight matrix (paper
Sec. 3.1: each row is split into blocks of length L).  The matrices stand in
for incoherence-processed (approximately iid Gaussian) Llama-3.2-1B
projection weights; none of the paper's models or datasets are used.

Seeds: 1000 * cfg + {0: codebook, 1: weights, 2 + call: upstream gradient,
500: [S, 2] codebook of the vector-emission trellis, 600: calibration inputs,
900: parity subset}.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    state_bits: int
    k: int
    L: int
    rows: int
    cols: int
    temps: tuple
    weights: str          # "normal", "normal_rms_block", "student5"
    outputs: tuple        # subset of ("w_soft", "logZ", "dW", "dc", "viterbi")

    @property
    def S(self) -> int:
        return 1 << self.state_bits

    @property
    def B(self) -> int:
        return self.rows * self.cols // self.L

    @property
    def edges(self) -> int:
        """Trellis edges per call: B * L * S * 2^k."""
        return self.B * self.L * self.S * (1 << self.k)


def anneal_temperatures(t0=0.1, t_end=1e-3, calls=8):
    """Geometric schedule T_i = t0 (t_end / t0)^(i / (calls - 1)), i = 0..calls-1
    (the exponential schedule of paper Sec. 3.6, sampled at both ends)."""
    return tuple(float(t0 * (t_end / t0) ** (i / (calls - 1))) for i in range(calls))


WORKLOADS = {
    1: Workload(1, "tiny S=16 k=2 L=16 B=64", 4, 2, 16, 64, 16, (1.0, 0.1, 1e-4), "normal",
                ("w_soft", "logZ", "dW", "dc", "viterbi")),
    2: Workload(2, "small S=256 k=2 L=256 1024x1024", 8, 2, 256, 1024, 1024, (1.0, 0.1, 0.01),
                "normal_rms_block", ("w_soft", "logZ", "dW")),
    3: Workload(3, "mid S=4096 k=2 L=256 2048x2048 student-t5", 12, 2, 256, 2048, 2048, (0.1,),
                "student5", ("w_soft", "logZ", "dW", "dc")),
    4: Workload(4, "full S=65536 k=2 L=256 2048x2048 (q/o-proj shape)", 16, 2, 256, 2048, 2048,
                (0.05,), "normal", ("w_soft", "logZ", "dW")),
    5: Workload(5, "full S=65536 k=2 L=256 2048x8192 (gate/up-proj shape), 8-call anneal", 16, 2,
                256, 2048, 8192, anneal_temperatures(), "normal",
                ("w_soft", "logZ", "dW", "dc", "viterbi")),
}


def workload(cfg: int) -> Workload:
    return WORKLOADS[cfg]


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def codebook(cfg: int) -> np.ndarray:
    wl = WORKLOADS[cfg]
    return _rng(1000 * cfg + 0).standard_normal(wl.S).astype(np.float32)


def weights(cfg: int, rows: int | None = None) -> np.ndarray:
    """Weights as [B, L] float32.  ``rows`` keeps only the first rows of the
    matrix (same values as the full draw for those rows)."""
    wl = WORKLOADS[cfg]
    r = _rng(1000 * cfg + 1)
    nrows = wl.rows if rows is None else rows
    if wl.weights == "normal":
        W = r.standard_normal((wl.rows, wl.cols))[:nrows]
    elif wl.weights == "normal_rms_block":
        W = 0.02 * r.standard_normal((wl.rows, wl.cols))[:nrows]
    elif wl.weights == "student5":
        W = r.standard_t(5, size=(wl.rows, wl.cols))[:nrows] * np.sqrt(3.0 / 5.0)
    else:  # pragma: no cover
        raise ValueError(wl.weights)
    W = W.reshape(-1, wl.L)
    if wl.weights == "normal_rms_block":
        W = W / np.sqrt((W * W).mean(axis=1, keepdims=True))
    return np.ascontiguousarray(W, dtype=np.float32)


def codebook_vec(cfg: int, V: int = 2) -> np.ndarray:
    """A [S, V] N(0,1) codebook for the vector-emission trellis (seed
    1000 * cfg + 500)."""
    wl = WORKLOADS[cfg]
    return _rng(1000 * cfg + 500).standard_normal((wl.S, V)).astype(np.float32)


def calibration_inputs(cfg: int, n_x: int = 4096) -> np.ndarray:
    """Synthetic layer inputs X [n_x, cols] for a proxy Hessian H = X^T X / n_x:
    N(0,1) draws times per-column scales exp(N(0, 0.5^2)), the uneven input
    channel energies of LLM activations (seed 1000 * cfg + 600)."""
    wl = WORKLOADS[cfg]
    r = _rng(1000 * cfg + 600)
    scale = np.exp(0.5 * r.standard_normal(wl.cols)).astype(np.float32)
    X = r.standard_normal((n_x, wl.cols), dtype=np.float32)
    return X * scale[None, :]


def upstream(cfg: int, call: int = 0, B: int | None = None) -> np.ndarray:
    wl = WORKLOADS[cfg]
    r = _rng(1000 * cfg + 2 + call)
    g = r.standard_normal((wl.B, wl.L))
    if B is not None:
        g = g[:B]
    return np.ascontiguousarray(g, dtype=np.float32)


def parity_subset(cfg: int, count: int = 64) -> np.ndarray:
    """Seeded sorted choice of block indices for checks at full size."""
    wl = WORKLOADS[cfg]
    return np.sort(_rng(1000 * cfg + 900).choice(wl.B, size=min(count, wl.B), replace=False))


def random_case(seed: int, B: int, L: int, state_bits: int, scale: float = 1.0):
    """Generic small case: (w[B,L], c[S], g[B,L]) float32, all N(0, scale^2)."""
    r = _rng(seed)
    c = (scale * r.standard_normal(1 << state_bits)).astype(np.float32)
    w = (scale * r.standard_normal((B, L))).astype(np.float32)
    g = r.standard_normal((B, L)).astype(np.float32)
    return w, c, g

"""GPU checks of the training helpers and the annealing loop against the
oracle and the published update formulas.

  computed codebook   within one fp32 ulp of the oracle's fp64 quantiles
                      (scipy ndtri) under the same permutation
  Adam / SGD kernels  within 2e-6 relative of the formulas evaluated in fp64
  annealing loop      plain-gradient runs follow the loop driven by the fp64
                      oracle VJP: |W_gpu - W_ref| <= 1e-3 max|W_ref - W_init|
                      (the VJP tolerance, 1e-4, accumulated over the steps);
                      the clipped drift stays within lr * N * g_max; the final
                      snap is the oracle's Viterbi codeword of the final W
"""
import sys

import numpy as np
import pytest

import paper_2605_10655_amd as P
from oracle import oracle as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


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


@pytest.mark.parametrize("n,V,seed", [(4, 1, 0), (8, 2, 3), (12, 1, 99), (16, 1, 7), (16, 2, 2605)])
def test_gaussian_codebook_matches_oracle(n, V, seed):
    _say(f"[qat] codebook n={n} V={V} seed={seed}")
    c = host(P.bcjr_gaussian_codebook(n, V, seed))
    ref = np.asarray(O.gaussian_codebook(n, V, seed), np.float64).reshape(c.shape).astype(np.float32)
    ulps = np.abs(c.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
    assert ulps.max() <= 1, ulps.max()


def test_adam_and_sgd_kernels_match_the_formulas():
    r = np.random.default_rng(1)
    p0 = r.standard_normal(10007).astype(np.float32)
    gs = [r.standard_normal(10007).astype(np.float32) * 3 for _ in range(4)]
    lr, b1, b2, eps, clip = 1e-2, 0.9, 0.999, 1e-8, 2.0
    p, m, v = dev(p0), torch.zeros(10007, device="cuda:0"), torch.zeros(10007, device="cuda:0")
    pr, mr, vr = p0.astype(np.float64), np.zeros(10007), np.zeros(10007)
    for step, g in enumerate(gs, start=1):
        P.qat_adam_step(p, dev(g), m, v, lr, b1, b2, eps, step, clip)
        gc = np.clip(g.astype(np.float64), -clip, clip)
        mr = b1 * mr + (1 - b1) * gc
        vr = b2 * vr + (1 - b2) * gc * gc
        pr = pr - lr * (mr / (1 - b1 ** step)) / (np.sqrt(vr / (1 - b2 ** step)) + eps)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(p), pr, rtol=2e-6, atol=2e-6)
    q = dev(p0)
    P.qat_sgd_step(q, dev(gs[0]), 0.05, 1.0)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(q), p0 - 0.05 * np.clip(gs[0], -1, 1), rtol=1e-6, atol=1e-7)


def _oracle_loop(W0, c, n, k, temps, lr, clip, block, learn=False, lr_c=0.0):
    """The annealing loop with plain gradient steps, in fp64 on the CPU."""
    W = W0.astype(np.float64)
    cc = np.asarray(c, np.float64).copy()
    for T in temps:
        Wb = W.reshape(-1, block)
        ws, _ = O.soft_codeword(Wb, cc, n, k, T)
        G = 2.0 * (ws.reshape(W.shape) - W0)
        _, _, dW, dc = O.soft_codeword_vjp(Wb, cc, n, k, T, G.reshape(-1, block))
        W = W - lr * np.clip(dW.reshape(W.shape), -clip, clip)
        if learn:
            cc = cc - lr_c * dc
    return W, cc


@pytest.mark.parametrize("learn", [False, True])
def test_annealing_loop_follows_the_oracle(learn):
    from paper_2605_10655_amd.qat import QATConfig, anneal_qat
    n, k, block = 8, 2, 32
    r = np.random.default_rng(5)
    W0 = r.standard_normal((16, 64)).astype(np.float32)
    c = r.standard_normal(1 << n).astype(np.float32)
    cfg = QATConfig(state_bits=n, k=k, block=block, T0=0.5, T_end=0.05, steps=5, lr=0.02,
                    grad_clip=0.5, optimizer="sgd", learn_codebook=learn, lr_codebook=0.01)
    _say(f"[qat] loop learn={learn}")
    res = anneal_qat(dev(W0), dev(c), cfg)
    torch.cuda.synchronize()
    temps = [float(np.float32(T)) for T in res.temps]
    Wr, cr = _oracle_loop(W0, c, n, k, temps, cfg.lr, cfg.grad_clip, block, learn, cfg.lr_codebook)
    scale = np.abs(Wr - W0).max()
    err = np.abs(host(res.W) - Wr).max()
    _say(f"[qat] loop learn={learn} drift {scale:.3e} err {err:.3e}")
    assert err <= 1e-3 * scale + 1e-6
    if learn:
        cs = np.abs(cr - c).max()
        assert np.abs(host(res.codebook) - cr).max() <= 1e-3 * cs + 1e-6
    # drift budget: clipped plain steps move no weight by more than lr * N * g_max
    assert res.max_drift <= cfg.lr * cfg.steps * cfg.grad_clip * (1 + 1e-6)
    # the snap is the Viterbi codeword of the final pre-image
    st, _ = O.viterbi(host(res.W).reshape(-1, block), host(res.codebook), n, k)
    np.testing.assert_array_equal(host(res.W_hard).reshape(-1, block), host(res.codebook)[st])


def test_annealing_loop_variants_run():
    """Adam, BCJR-STE, the vector trellis and a proxy Hessian through the
    same loop: finite losses, the drift within the Adam step bound."""
    from paper_2605_10655_amd.qat import QATConfig, anneal_qat
    r = np.random.default_rng(6)
    W0 = dev(r.standard_normal((8, 128)).astype(np.float32))
    X = r.standard_normal((64, 128)).astype(np.float32)
    H = dev((X.T @ X / 64).astype(np.float32))
    c1 = P.bcjr_gaussian_codebook(10, 1, 1)
    c2 = P.bcjr_gaussian_codebook(12, 2, 1)
    runs = [
        (QATConfig(state_bits=10, k=2, block=64, T0=0.2, T_end=0.005, steps=6, lr=0.01), c1, None),
        (QATConfig(state_bits=10, k=2, block=64, T0=0.2, T_end=0.005, steps=6, lr=0.01, ste=True,
                   learn_codebook=True), c1, H),
        (QATConfig(state_bits=12, k=4, V=2, block=64, T0=0.2, T_end=0.05, steps=4, lr=0.01), c2, H),
    ]
    for cfg, c, Hm in runs:
        _say(f"[qat] variant ste={cfg.ste} V={cfg.V} H={Hm is not None}")
        res = anneal_qat(W0, c, cfg, H=Hm)
        torch.cuda.synchronize()
        assert all(np.isfinite(res.losses)) and np.isfinite(res.loss_hard)
        # Adam moves a weight by at most about lr per step (|m_hat| / sqrt(v_hat) <= 1 here)
        assert res.max_drift <= 1.5 * cfg.lr * cfg.steps

"""GPU checks of the BlockLDLQ trellis rounding against the oracle.

  each column block's decode is the oracle's Viterbi path of the same
  fp32 target, bit-exact;
  the targets match the fp64 feedback formula evaluated on the GPU's own
  rounding within 1e-5 of the weights' scale;
  the Hessian-weighted loss of the result is within 1e-3 of the oracle's
  and below that of the plain per-block Viterbi codeword.
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


def _case(seed, rows, cols, n, V=1):
    r = np.random.default_rng(seed)
    W = r.standard_normal((rows, cols)).astype(np.float32)
    c = r.standard_normal((1 << n) * V).astype(np.float32)
    X = r.standard_normal((4 * cols, cols)) @ (np.eye(cols) + 0.7 * r.standard_normal((cols, cols)) / np.sqrt(cols))
    H = (X.T @ X / (4 * cols)).astype(np.float32)
    return W, c, H


@pytest.mark.parametrize("n,k,V,rows,cols,block", [
    (8, 2, 1, 16, 128, 32), (12, 2, 1, 8, 256, 64), (8, 4, 2, 12, 96, 32), (16, 2, 1, 4, 512, 256),
])
def test_ldlq_matches_oracle(n, k, V, rows, cols, block):
    from paper_2605_10655_amd.ldlq import hw_loss, ldlq_viterbi
    W, c, H = _case(n * 100 + cols, rows, cols, n, V)
    cb = c.reshape(-1, V) if V > 1 else c
    _say(f"[ldlq] n={n} k={k} V={V} {rows}x{cols} block={block}")
    Wh, st, tg = ldlq_viterbi(dev(W), dev(cb), n, k, dev(H), block=block, V=V, return_targets=True)
    torch.cuda.synchronize()
    Wh, st, tg = host(Wh), host(st), host(tg)
    for j in range(cols // block):
        ref, _ = O.viterbi(tg[j], cb, n, k, V=V)
        np.testing.assert_array_equal(st[j], ref)
    _, _, tref = O.ldlq_viterbi(W, cb, n, k, H, block, V=V, targets_from=Wh)
    assert np.abs(tg - tref).max() <= 1e-5 * max(1.0, np.abs(W).max())
    Wo, _, _ = O.ldlq_viterbi(W, cb, n, k, H, block, V=V)
    l_gpu = hw_loss(torch.from_numpy(W), torch.from_numpy(Wh), torch.from_numpy(H))
    l_ref = hw_loss(torch.from_numpy(W), torch.from_numpy(Wo.astype(np.float32)), torch.from_numpy(H))
    st_plain, _ = O.viterbi(W.reshape(-1, block), cb, n, k, V=V)
    plain = np.asarray(cb).reshape(-1, V)[st_plain].reshape(W.shape)
    l_plain = hw_loss(torch.from_numpy(W), torch.from_numpy(plain.astype(np.float32)), torch.from_numpy(H))
    _say(f"[ldlq] loss gpu {l_gpu:.4f} oracle {l_ref:.4f} plain {l_plain:.4f}")
    assert abs(l_gpu - l_ref) <= 1e-3 * l_ref
    assert l_gpu < l_plain


@pytest.mark.parametrize("d,block,damp", [(96, 32, 0.0), (128, 32, 0.01), (256, 64, 0.01),
                                          (512, 256, 0.01), (80, 16, 0.05)])
def test_block_ldl_matches_oracle(d, block, damp):
    """The device factorisation (fp64 Cholesky of the index-reversed damped
    Hessian, per-block inverses) against the oracle's numpy block_ldl of the
    same damped matrix, and M D M^T = H + damp mean(diag H) I."""
    from paper_2605_10655_amd.ldlq import block_ldl
    _, _, H = _case(d + block, 4, d, 8)
    _say(f"[ldl] d={d} block={block} damp={damp}")
    M, D = block_ldl(dev(H), block, damp)
    torch.cuda.synchronize()
    M, D = host(M), host(D)
    Hd = H.astype(np.float64)
    Hd = Hd + damp * np.mean(np.diag(Hd)) * np.eye(d)
    Mr, Dr = O.block_ldl(Hd, block)
    scale = np.abs(Mr).max()
    assert np.abs(M - Mr).max() <= 1e-9 * scale, np.abs(M - Mr).max()
    assert np.abs(D - Dr).max() <= 1e-9 * np.abs(Dr).max()
    assert np.abs(M @ D @ M.T - Hd).max() <= 1e-9 * np.abs(Hd).max()
    for kb in range(0, d, block):          # unit diagonal blocks, zero below them
        np.testing.assert_allclose(M[kb:kb + block, kb:kb + block], np.eye(block), atol=1e-9)
        assert np.all(M[kb + block:, kb:kb + block] == 0.0)

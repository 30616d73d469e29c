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

"""Pins for oracle.dense against things other than itself: an independent
library implementation (torch float64 softmax attention and autograd),
central finite differences, and closed-form special cases."""
import numpy as np
import pytest
import torch

from oracle import dense


def _rand(rng, B, L, H, d, scale=1.0):
    return [scale * rng.standard_normal((B, L, H, d)) for _ in range(4)]


def _torch_ref(Q, K, V, causal):
    """Independent float64 reference: torch softmax attention with autograd."""
    q, k, v = (torch.tensor(x.transpose(0, 2, 1, 3), requires_grad=True) for x in (Q, K, V))
    d = Q.shape[-1]
    s = (q @ k.transpose(-1, -2)) / np.sqrt(d)
    if causal:
        L = Q.shape[1]
        s = s.masked_fill(~torch.ones(L, L, dtype=torch.bool).tril(), float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    o = torch.softmax(s, dim=-1) @ v
    return q, k, v, o, lse


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("shape", [(1, 1, 1, 4), (2, 37, 3, 16), (1, 130, 2, 64)])
def test_forward_matches_torch(causal, shape):
    rng = np.random.default_rng(1)
    Q, K, V, _ = _rand(rng, *shape)
    O, LSE = dense.attention_forward(Q, K, V, causal)
    _, _, _, o, lse = _torch_ref(Q, K, V, causal)
    np.testing.assert_allclose(O, o.detach().numpy().transpose(0, 2, 1, 3), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(LSE, lse.detach().numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_backward_matches_torch_autograd(causal):
    rng = np.random.default_rng(2)
    Q, K, V, dO = _rand(rng, 2, 45, 2, 16)
    dQ, dK, dV, O, LSE = dense.attention_backward(Q, K, V, dO, causal)
    q, k, v, o, lse = _torch_ref(Q, K, V, causal)
    o.backward(torch.tensor(dO.transpose(0, 2, 1, 3)))
    tr = lambda t: t.detach().numpy().transpose(0, 2, 1, 3)
    np.testing.assert_allclose(dQ, tr(q.grad), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dK, tr(k.grad), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, tr(v.grad), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(O, tr(o), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(LSE, lse.detach().numpy(), rtol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_backward_finite_differences(causal):
    """Central differences of loss = sum(O * W) at L <= 64 in float64."""
    rng = np.random.default_rng(3)
    B, L, H, d = 1, 24, 2, 8
    Q, K, V, W = _rand(rng, B, L, H, d)
    dQ, dK, dV, _, _ = dense.attention_backward(Q, K, V, W, causal)
    eps = 1e-6
    loss = lambda Q_, K_, V_: float((dense.attention_forward(Q_, K_, V_, causal)[0] * W).sum())
    for name, X, G in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        idx = [tuple(rng.integers(0, s) for s in X.shape) for _ in range(12)]
        for i in idx:
            Xp = X.copy(); Xp[i] += eps
            Xm = X.copy(); Xm[i] -= eps
            args_p = {"Q": (Xp, K, V), "K": (Q, Xp, V), "V": (Q, K, Xp)}[name]
            args_m = {"Q": (Xm, K, V), "K": (Q, Xm, V), "V": (Q, K, Xm)}[name]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - G[i]) < 1e-7, (name, i, fd, G[i])


def test_zero_query_gives_mean_and_prefix_mean():
    rng = np.random.default_rng(4)
    B, L, H, d = 1, 19, 2, 8
    Q = np.zeros((B, L, H, d)); K = rng.standard_normal((B, L, H, d)); V = rng.standard_normal((B, L, H, d))
    O, LSE = dense.attention_forward(Q, K, V, causal=False)
    np.testing.assert_allclose(O, np.broadcast_to(V.mean(axis=1, keepdims=True), O.shape), atol=1e-14)
    np.testing.assert_allclose(LSE, np.log(L), atol=1e-14)
    O, LSE = dense.attention_forward(Q, K, V, causal=True)
    prefix = np.cumsum(V, axis=1) / np.arange(1, L + 1)[None, :, None, None]
    np.testing.assert_allclose(O, prefix, atol=1e-14)
    np.testing.assert_allclose(LSE[0, 0], np.log(np.arange(1, L + 1)), atol=1e-14)


def test_constant_value_and_single_token():
    rng = np.random.default_rng(5)
    Q, K, _, _ = _rand(rng, 2, 9, 3, 4)
    V = np.broadcast_to(rng.standard_normal((2, 1, 3, 4)), (2, 9, 3, 4)).copy()
    O, _ = dense.attention_forward(Q, K, V, causal=True)
    np.testing.assert_allclose(O, V, atol=1e-14)
    Q, K, V, _ = _rand(rng, 1, 1, 1, 16)
    O, LSE = dense.attention_forward(Q, K, V, causal=False)
    np.testing.assert_allclose(O, V, atol=1e-15)
    np.testing.assert_allclose(LSE[0, 0, 0], (Q[0, 0, 0] @ K[0, 0, 0]) / 4.0, rtol=1e-14)


def test_row_subsets_and_per_head_rows():
    rng = np.random.default_rng(6)
    Q, K, V, _ = _rand(rng, 1, 70, 2, 8)
    O, LSE = dense.attention_forward(Q, K, V, causal=True)
    rows = np.array([0, 5, 33, 69])
    Os, LSEs = dense.attention_forward(Q, K, V, causal=True, rows=rows, row_chunk=3)
    # a row subset in chunks of 3 rows hands BLAS other matrix shapes than the
    # full call, so its blocking, and the float64 summation order of each dot
    # product, differ: equal up to a few ulps of the sums (rtol 1e-12), not to
    # the last bit
    np.testing.assert_allclose(Os, O[:, rows], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(LSEs, LSE[:, :, rows], rtol=1e-12, atol=1e-14)
    per = [np.array([1, 2, 68]), np.array([0, 40, 69])]
    Op, LSEp = dense.attention_forward(Q, K, V, causal=True, rows=per)
    for h in range(2):
        np.testing.assert_allclose(Op[:, :, h], O[:, per[h], h], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(LSEp[:, h], LSE[:, h, per[h]], rtol=1e-12, atol=1e-14)


def test_rel_l2():
    assert dense.rel_l2(np.array([3.0, 4.0]), np.array([3.0, 4.0])) == 0.0
    assert abs(dense.rel_l2(np.array([3.0, 5.0]), np.array([3.0, 4.0])) - 0.2) < 1e-15


@pytest.mark.parametrize("causal", [False, True])
def test_backward_rows_equal_the_full_backward(causal):
    """attention_backward_rows (sampled query rows for dQ, sampled key rows
    for dK and dV, one pass over query chunks) against the full-matrix
    attention_backward, itself pinned by autograd and finite differences."""
    rng = np.random.default_rng(11)
    Q, K, V, dO = _rand(rng, 2, 70, 3, 8)
    gQ, gK, gV, _, _ = dense.attention_backward(Q, K, V, dO, causal)
    qr, kr = np.array([0, 9, 33, 69]), np.array([0, 1, 50, 68, 69])
    dQ, dK, dV = dense.attention_backward_rows(Q, K, V, dO, causal, qr, kr, row_chunk=16)
    np.testing.assert_allclose(dQ, gQ[:, qr], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(dK, gK[:, kr], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(dV, gV[:, kr], rtol=1e-11, atol=1e-13)
    per_q = [np.array([3, 4]), np.array([0, 69]), np.array([10, 20])]
    per_k = [np.array([69, 5]), np.array([7, 8]), np.array([0, 1])]
    dQ, dK, dV = dense.attention_backward_rows(Q, K, V, dO, causal, per_q, per_k, row_chunk=7)
    for h in range(3):
        np.testing.assert_allclose(dQ[:, :, h], gQ[:, per_q[h], h], rtol=1e-11, atol=1e-13)
        np.testing.assert_allclose(dK[:, :, h], gK[:, per_k[h], h], rtol=1e-11, atol=1e-13)
        np.testing.assert_allclose(dV[:, :, h], gV[:, per_k[h], h], rtol=1e-11, atol=1e-13)

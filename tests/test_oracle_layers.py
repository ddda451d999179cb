"""Pins for the oracle's layer math (CPU only).

Each layer primitive of the oracle is checked against an independent
library routine (torch CPU ops in float64 with autograd) and against
closed forms and invariants of the operation itself.  Nothing here touches
the GPU library.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle



def _t(a, grad=False):
    return torch.tensor(np.asarray(a, dtype=np.float64), dtype=torch.float64, requires_grad=grad)


CONV_CASES = [
    # N, Ci, H, W, Co, R, stride, pad, bias
    (2, 3, 9, 7, 5, 3, 1, 1, False),
    (2, 4, 10, 10, 6, 3, 2, 1, False),
    (1, 1, 12, 12, 6, 5, 1, 2, True),
    (3, 6, 14, 14, 16, 5, 1, 0, True),
    (2, 8, 9, 9, 4, 1, 2, 0, False),
    (2, 3, 16, 16, 8, 7, 2, 3, False),
    (2, 5, 6, 6, 7, 1, 1, 0, True),
]


@pytest.mark.parametrize("N,Ci,H,W,Co,R,st,pad,bias", CONV_CASES)
def test_conv_matches_torch(oracle_lib, N, Ci, H, W, Co, R, st, pad, bias):
    rng = np.random.default_rng(N * 1000 + Ci * 100 + R)
    x = rng.standard_normal((N, Ci, H, W))
    w = rng.standard_normal((Co, Ci, R, R))
    b = rng.standard_normal(Co) if bias else None
    Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    dy = rng.standard_normal((N, Co, Ho, Wo))
    y, dx, dw, db = oracle.conv2d(x, w, b, st, pad, dy=dy)
    xt, wt = _t(x, True), _t(w, True)
    bt = _t(b, True) if bias else None
    yt = F.conv2d(xt, wt, bt, stride=st, padding=pad)
    yt.backward(_t(dy))
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-12, atol=1e-11)
    if bias:
        np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-11)


def test_conv_delta_kernel_is_shift(oracle_lib):
    """A kernel with a single 1 at tap (r, s) copies the input shifted by
    (r - pad, s - pad): a closed form of the convolution sum."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((1, 1, 6, 6))
    w = np.zeros((1, 1, 3, 3))
    w[0, 0, 2, 0] = 1.0
    y, *_ = oracle.conv2d(x, w, None, 1, 1)
    xp = np.pad(x[0, 0], 1)
    np.testing.assert_array_equal(y[0, 0], xp[2:8, 0:6])


def test_batchnorm_matches_torch_and_invariants(oracle_lib):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((4, 5, 3, 3)) * 3.0 + 1.5
    g = rng.standard_normal(5)
    b = rng.standard_normal(5)
    dy = rng.standard_normal(x.shape)
    y, dx, dg, dbt = oracle.batchnorm(x, g, b, dy=dy)
    xt, gt, bt = _t(x, True), _t(g, True), _t(b, True)
    yt = F.batch_norm(xt, None, None, gt, bt, training=True, eps=1e-5)
    yt.backward(_t(dy))
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-12, atol=1e-11)
    np.testing.assert_allclose(dbt, bt.grad.numpy(), rtol=1e-12, atol=1e-11)
    # gamma=1, beta=0: each channel has mean 0 and variance var/(var+eps)
    y1, dx1, _, _ = oracle.batchnorm(x, np.ones(5), np.zeros(5), dy=dy)
    var = x.var(axis=(0, 2, 3))
    np.testing.assert_allclose(y1.mean(axis=(0, 2, 3)), 0.0, atol=1e-13)
    np.testing.assert_allclose(y1.var(axis=(0, 2, 3)), var / (var + 1e-5), rtol=1e-12)
    # the input gradient sums to zero over each channel
    np.testing.assert_allclose(dx1.sum(axis=(0, 2, 3)), 0.0, atol=1e-11)


@pytest.mark.parametrize("K,st,pad", [(2, 2, 0), (3, 2, 1)])
def test_maxpool_matches_torch(oracle_lib, K, st, pad):
    rng = np.random.default_rng(3 + K)
    x = rng.standard_normal((2, 3, 8, 8))
    Ho = (8 + 2 * pad - K) // st + 1
    dy = rng.standard_normal((2, 3, Ho, Ho))
    y, dx = oracle.maxpool(x, K, st, pad, dy=dy)
    xt = _t(x, True)
    yt = F.max_pool2d(xt, K, st, pad)
    yt.backward(_t(dy))
    np.testing.assert_array_equal(y, yt.detach().numpy())
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=0, atol=1e-15)


def test_maxpool_tie_takes_first_cell(oracle_lib):
    x = np.zeros((1, 1, 2, 2))
    y, dx = oracle.maxpool(x, 2, 2, 0, dy=np.ones((1, 1, 1, 1)))
    assert dx[0, 0].tolist() == [[1.0, 0.0], [0.0, 0.0]]


def test_softmax_xent(oracle_lib):
    rng = np.random.default_rng(4)
    o = rng.standard_normal((6, 10)) * 4
    y = rng.integers(0, 10, 6)
    loss, d = oracle.softmax_xent(o, y)
    ot = _t(o, True)
    lt = F.cross_entropy(ot, torch.tensor(y, dtype=torch.long))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-13
    np.testing.assert_allclose(d, ot.grad.numpy(), atol=1e-15)
    # closed form: gradient rows are (softmax - onehot)/N and sum to zero
    np.testing.assert_allclose(d.sum(axis=1), 0.0, atol=1e-15)
    # uniform logits: loss = ln(classes)
    l0, d0 = oracle.softmax_xent(np.full((3, 1000), 0.25), np.array([0, 5, 999]))
    assert abs(l0 - np.log(1000)) < 1e-12
    assert abs(d0[1, 5] - (1 / 1000 - 1) / 3) < 1e-15
    # a huge logit gap does not overflow (max-subtracted log-sum-exp)
    l1, _ = oracle.softmax_xent(np.array([[1000.0, 0.0]]), np.array([1]))
    assert abs(l1 - 1000.0) < 1e-9


@pytest.mark.parametrize("N,Ci,H,W,Co,R,st,pad,bias", CONV_CASES)
def test_conv_samples_match_loop_formulation(oracle_lib, N, Ci, H, W, Co, R, st, pad, bias):
    """Two formulations inside the oracle: whole-tensor loops and one
    element at a time from the definition."""
    rng = np.random.default_rng(7 + R)
    x = rng.standard_normal((N, Ci, H, W)).astype(np.float32)
    w = rng.standard_normal((Co, Ci, R, R)).astype(np.float32)
    b = rng.standard_normal(Co).astype(np.float32) if bias else None
    Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    dy = rng.standard_normal((N, Co, Ho, Wo)).astype(np.float32)
    y, dx, dw, db = oracle.conv2d(x, w, b, st, pad, dy=dy)
    geo = dict(N=N, Ci=Ci, H=H, W=W, Co=Co, R=R, stride=st, pad=pad)
    qy = np.stack(np.meshgrid(*[np.arange(d) for d in y.shape], indexing="ij"), -1).reshape(-1, 4)
    np.testing.assert_allclose(oracle.conv_samples(0, qy, x=x, w=w, bias=b, **geo),
                               y.reshape(-1), rtol=1e-12, atol=1e-12)
    qw = np.stack(np.meshgrid(*[np.arange(d) for d in w.shape], indexing="ij"), -1).reshape(-1, 4)
    np.testing.assert_allclose(oracle.conv_samples(1, qw, x=x, dy=dy, **geo), dw.reshape(-1),
                               rtol=1e-12, atol=1e-11)
    qx = np.stack(np.meshgrid(*[np.arange(d) for d in x.shape], indexing="ij"), -1).reshape(-1, 4)
    np.testing.assert_allclose(oracle.conv_samples(2, qx, dy=dy, w=w, **geo), dx.reshape(-1),
                               rtol=1e-12, atol=1e-11)

"""Pins for the oracle's SMA update, Algorithm 1 (Sec. 3.2), CPU only.

None of these restates the update: each checks an identity or a special
case that Algorithm 1 must satisfy and that a plausible slip (gradient and
correction taken at different points, a sign, a dropped momentum term, the
wrong z_prev) breaks:

* alpha = 1/k makes the new z the replicas' mean plus the momentum term;
* the corrections added to z equal those removed from the replicas;
* mu = 0 is synchronous elastic averaging (the EA-SGD comparison of
  Sec. 5.5) with period 1;
* k = 1, alpha = 0 is plain SGD (Eq. 1) -- or heavy-ball momentum (Eq. 3)
  when learner momentum is on -- in closed form on a quadratic, z fixed;
* identical replicas at zero velocity with zero gradient do not move;
* alpha = 0 decouples the learners: each equals an independent k = 1 run;
* permuting learners permutes replicas and leaves z unchanged;
* on a shared quadratic the iteration converges to its minimiser.
"""
import numpy as np
import pytest

import oracle
import workloads as wl

LENET = ("lenet5", 1, 28, 28, 10)


def _ctx(k, P_model=LENET, alpha=None, lr=0.05, mu=0.9, mu_l=0.0, b=2, seed=0):
    m = oracle.model(*P_model)
    w0 = wl.init_w0(oracle.tensors(m), seed)
    return oracle.SMA(m, w0, k, b, 1.0 / k if alpha is None else alpha, lr, mu, mu_l), w0


def _random_state(c, rng, same=False):
    P, k = c.P, c.k
    W = rng.standard_normal((k, P)) * 0.1
    if same:
        W[:] = W[0]
    Z = rng.standard_normal(P) * 0.1
    Zp = Z + rng.standard_normal(P) * 0.01
    c.set_state(W, Z, Zp)
    return W, Z, Zp


@pytest.mark.parametrize("k", [1, 2, 3, 8])
def test_alpha_one_over_k_gives_mean_plus_momentum(oracle_lib, k):
    rng = np.random.default_rng(k)
    c, _ = _ctx(k, lr=0.05, mu=0.9)
    W, Z, Zp = _random_state(c, rng)
    G = rng.standard_normal((k, c.P))
    c.sma_apply(G)
    np.testing.assert_allclose(c.central(), W.mean(axis=0) + 0.9 * (Z - Zp), rtol=0, atol=1e-14)
    np.testing.assert_array_equal(c.prev_central(), Z)


@pytest.mark.parametrize("k,alpha,mu", [(4, 0.25, 0.9), (3, 0.1, 0.5), (5, 0.7, 0.0)])
def test_corrections_are_conserved(oracle_lib, k, alpha, mu):
    rng = np.random.default_rng(10 + k)
    lr = 0.03
    c, _ = _ctx(k, alpha=alpha, lr=lr, mu=mu)
    W, Z, Zp = _random_state(c, rng)
    G = rng.standard_normal((k, c.P))
    c.sma_apply(G)
    Wn = np.stack([c.replica(j) for j in range(k)])
    removed = (W - lr * G - Wn).sum(axis=0)
    added = c.central() - Z - mu * (Z - Zp)
    np.testing.assert_allclose(removed, added, rtol=0, atol=1e-13)


def test_mu_zero_is_elastic_averaging(oracle_lib):
    """EA-SGD with period 1: x_i <- x_i - g_i - a(x_i - x~),
    x~ <- x~ + a * sum_i (x_i - x~), both from the old values."""
    rng = np.random.default_rng(3)
    k, a, lr = 4, 0.2, 0.1
    c, _ = _ctx(k, alpha=a, lr=lr, mu=0.0)
    x, xt, _ = _random_state(c, rng)
    for _ in range(5):
        g = rng.standard_normal((k, c.P))
        c.sma_apply(g)
        x, xt = x - lr * g - a * (x - xt), xt + a * (x - xt).sum(axis=0)
    np.testing.assert_allclose(c.central(), xt, atol=1e-13)
    for j in range(k):
        np.testing.assert_allclose(c.replica(j), x[j], atol=1e-13)


@pytest.mark.parametrize("mu_l", [0.0, 0.9])
def test_single_learner_no_correction_is_sgd_closed_form(oracle_lib, mu_l):
    """k=1, alpha=0 on the quadratic 1/2 (w - a)^2 (gradient w - a).
    mu_l = 0: Eq. 1, e_n = (1 - lr)^n e_0.  mu_l = mu: Eq. 3, whose error
    obeys e_{n+1} = (1 - lr + mu) e_n - mu e_{n-1} with e_{-1} = e_0; its
    closed form is a power of the 2x2 companion matrix."""
    lr, mu, T = 0.1, 0.9, 30
    c, w0 = _ctx(1, alpha=0.0, lr=lr, mu=mu, mu_l=mu_l)
    rng = np.random.default_rng(4)
    a = rng.standard_normal(c.P)
    w = w0.astype(np.float64)
    for _ in range(T):
        c.sma_apply((c.replica(0) - a)[None, :])
    e0 = w - a
    if mu_l == 0.0:
        expect = a + (1 - lr) ** T * e0
    else:
        M = np.array([[1 - lr + mu_l, -mu_l], [1.0, 0.0]])
        coef = np.linalg.matrix_power(M, T) @ np.array([1.0, 1.0])
        expect = a + coef[0] * e0
    np.testing.assert_allclose(c.replica(0), expect, rtol=1e-11, atol=1e-12)
    # z never moves: no corrections, and z_prev starts equal to z (= w0)
    np.testing.assert_array_equal(c.central(), w)


def test_identical_replicas_zero_gradient_is_fixed_point(oracle_lib):
    k = 4
    c, w0 = _ctx(k, lr=0.1, mu=0.9)
    c.sma_apply(np.zeros((k, c.P)))
    np.testing.assert_array_equal(c.central(), w0.astype(np.float64))
    for j in range(k):
        np.testing.assert_array_equal(c.replica(j), w0.astype(np.float64))


def test_first_sync_has_no_momentum(oracle_lib):
    """z_prev starts at w0 (zero initial velocity), so the first sync moves
    z by exactly the sum of the corrections."""
    k = 2
    c, w0 = _ctx(k, lr=0.1, mu=0.9)
    rng = np.random.default_rng(5)
    G = rng.standard_normal((k, c.P))
    c.sma_apply(G)
    # at step 1 every replica equals z, so every correction is zero
    np.testing.assert_array_equal(c.central(), w0.astype(np.float64))
    c.sma_apply(G)
    W1 = w0.astype(np.float64) - 0.1 * G
    np.testing.assert_allclose(c.central(), W1.mean(axis=0), atol=1e-15)


def test_alpha_zero_decouples_learners(oracle_lib):
    """Learners only interact through the corrections: with alpha = 0 each
    replica of a k = 3 run equals a k = 1 run on that learner's images."""
    k, b, T = 3, 2, 3
    m = oracle.model(*LENET)
    w0 = wl.init_w0(oracle.tensors(m), 1)
    big = oracle.SMA(m, w0, k, b, 0.0, 0.05, 0.9)
    solo = [oracle.SMA(m, w0, 1, b, 0.0, 0.05, 0.9) for _ in range(k)]
    for t in range(T):
        x, y = wl.batch(k * b, 1, 28, 28, 10, seed=2, step=t)
        big.step(x, y)
        big.sync()
        for j in range(k):
            solo[j].step(x[j * b:(j + 1) * b], y[j * b:(j + 1) * b])
            solo[j].sync()
    for j in range(k):
        np.testing.assert_array_equal(big.replica(j), solo[j].replica(0))


def test_permuting_learners_permutes_replicas(oracle_lib):
    k, b = 3, 2
    m = oracle.model(*LENET)
    w0 = wl.init_w0(oracle.tensors(m), 2)
    perm = [2, 0, 1]
    A = oracle.SMA(m, w0, k, b, 1.0 / 3, 0.05, 0.9)
    B = oracle.SMA(m, w0, k, b, 1.0 / 3, 0.05, 0.9)
    for t in range(3):
        x, y = wl.batch(k * b, 1, 28, 28, 10, seed=3, step=t)
        idx = np.concatenate([np.arange(p * b, (p + 1) * b) for p in perm])
        A.step(x, y)
        A.sync()
        B.step(x[idx], y[idx])
        B.sync()
    for j in range(k):
        np.testing.assert_allclose(B.replica(j), A.replica(perm[j]), atol=1e-14)
    np.testing.assert_allclose(B.central(), A.central(), atol=1e-14)


def test_shared_quadratic_converges_to_minimiser(oracle_lib):
    k, lr, mu = 4, 0.1, 0.5
    c, _ = _ctx(k, lr=lr, mu=mu)
    rng = np.random.default_rng(6)
    a = rng.standard_normal(c.P)
    for _ in range(400):
        W = np.stack([c.replica(j) for j in range(k)])
        c.sma_apply(W - a)
    np.testing.assert_allclose(c.central(), a, atol=1e-9)
    np.testing.assert_allclose(c.replica(k - 1), a, atol=1e-9)


def test_unsynced_step_applies_local_update(oracle_lib):
    """Sync interval above one: a second step() without sync() first moves
    each replica by -lr * its pending gradient, with no correction."""
    k, b, lr = 2, 2, 0.05
    m = oracle.model(*LENET)
    w0 = wl.init_w0(oracle.tensors(m), 4)
    c = oracle.SMA(m, w0, k, b, 0.5, lr, 0.9)
    x, y = wl.batch(k * b, 1, 28, 28, 10, seed=4, step=0)
    c.step(x, y)
    g0 = [c.grad(j) for j in range(k)]
    x1, y1 = wl.batch(k * b, 1, 28, 28, 10, seed=4, step=1)
    c.step(x1, y1)
    for j in range(k):
        w1 = w0.astype(np.float64) - lr * g0[j]
        np.testing.assert_array_equal(c.replica(j), w1)
        _, gj = oracle.learner_grad(m, w1, x1[j * b:(j + 1) * b], y1[j * b:(j + 1) * b])
        np.testing.assert_array_equal(c.grad(j), gj)
    np.testing.assert_array_equal(c.central(), w0.astype(np.float64))
    assert c.sync() == 0
    assert c.sync() == -4  # nothing pending

"""Pins for the oracle's control operations around Algorithm 1, CPU only:
the learning-rate change and the restart of SMA (Sec. 3.2), resizing the
set of learners (Sec. 3.4, 4.4), and the decision rule of Algorithm 2.

* after a restart every replica and z_prev equal z, so a step with zero
  gradient moves nothing (without the reset of z_prev, z would still move
  by mu (z - z_prev));
* a new learning rate enters the replica update exactly where gamma does
  (checked on a quadratic with the alpha = 1/k mean identity);
* a learner added between iterations starts at z with zero velocity, takes
  part in the next correction sum, and the existing replicas are untouched;
  removing learners drops the newest ones;
* Algorithm 2 on hand-worked throughput sequences.
"""
import numpy as np
import pytest

import oracle
import workloads as wl

LENET = ("lenet5", 1, 28, 28, 10)


def _ctx(k, alpha=None, lr=0.05, mu=0.9, mu_l=0.0, b=2, seed=0):
    m = oracle.model(*LENET)
    w0 = wl.init_w0(oracle.tensors(m), seed)
    return oracle.SMA(m, w0, k, b, 1.0 / k if alpha is None else alpha, lr, mu, mu_l)


def _state(c, rng):
    W = rng.standard_normal((c.k, c.P)) * 0.1
    Z = rng.standard_normal(c.P) * 0.1
    Zp = Z + rng.standard_normal(c.P) * 0.01
    c.set_state(W, Z, Zp)
    return W, Z, Zp


@pytest.mark.parametrize("mu_l", [0.0, 0.9])
def test_restart_resets_replicas_and_velocity(oracle_lib, mu_l):
    rng = np.random.default_rng(1)
    c = _ctx(3, mu_l=mu_l)
    W, Z, Zp = _state(c, rng)
    c.restart()
    np.testing.assert_array_equal(c.prev_central(), Z)
    for j in range(3):
        np.testing.assert_array_equal(c.replica(j), Z)
    # zero gradient after a restart: a fixed point (z, z_prev, w_j, w_prev all z)
    c.sma_apply(np.zeros((3, c.P)))
    np.testing.assert_array_equal(c.central(), Z)
    for j in range(3):
        np.testing.assert_array_equal(c.replica(j), Z)


def test_restart_drops_a_pending_gradient(oracle_lib):
    c = _ctx(2, b=2)
    x, y = wl.batch(4, 1, 28, 28, 10, 0, 0)
    c.step(x, y)
    c.restart()
    assert c.sync() == -4  # nothing pending any more


def test_new_learning_rate_enters_where_gamma_does(oracle_lib):
    # alpha = 1/k: z' = mean(w) + mu (z - z_prev) does not involve gamma, and
    # each replica moves by -gamma g - alpha (w - z); compare the replica
    # change under two rates: the difference is exactly -(gamma2 - gamma1) g
    rng = np.random.default_rng(2)
    out = []
    for lr in (0.05, 0.2):
        c = _ctx(2, lr=0.05)
        W, Z, Zp = _state(c, np.random.default_rng(3))
        c.set_lr(lr)
        G = np.random.default_rng(4).standard_normal((2, c.P))
        c.sma_apply(G)
        out.append((c.replica(0), c.central(), G, W, Z, Zp))
    (r1, z1, G, W, Z, Zp), (r2, z2, _, _, _, _) = out
    np.testing.assert_allclose(r2 - r1, -(0.2 - 0.05) * G[0], rtol=0, atol=1e-14)
    np.testing.assert_allclose(z1, W.mean(axis=0) + 0.9 * (Z - Zp), rtol=0, atol=1e-14)
    np.testing.assert_array_equal(z1, z2)


def test_added_learner_starts_at_z_and_joins_the_average(oracle_lib):
    rng = np.random.default_rng(5)
    c = _ctx(2)
    W, Z, Zp = _state(c, rng)
    assert c.set_learners(3, 1.0 / 3) == 0
    for j in range(2):
        np.testing.assert_array_equal(c.replica(j), W[j])
    np.testing.assert_array_equal(c.replica(2), Z)
    G = rng.standard_normal((3, c.P))
    c.sma_apply(G)
    # alpha = 1/3 over three replicas, the new one at z
    Wn = np.vstack([W, Z[None]])
    np.testing.assert_allclose(c.central(), Wn.mean(axis=0) + 0.9 * (Z - Zp), rtol=0, atol=1e-14)
    # the new learner had zero velocity: with learner momentum off its step is
    # -gamma g - alpha (z - z) = -gamma g
    np.testing.assert_allclose(c.replica(2), Z - 0.05 * G[2], rtol=0, atol=1e-14)


def test_added_learner_has_zero_learner_velocity(oracle_lib):
    # with learner momentum the new replica's previous value is z too, so its
    # first update has no momentum term
    rng = np.random.default_rng(6)
    c = _ctx(1, mu_l=0.9)
    W, Z, Zp = _state(c, rng)
    assert c.set_learners(2, 0.0) == 0
    G = rng.standard_normal((2, c.P))
    c.sma_apply(G)
    np.testing.assert_allclose(c.replica(1), Z - 0.05 * G[1], rtol=0, atol=1e-14)


def test_removing_learners_keeps_the_oldest(oracle_lib):
    rng = np.random.default_rng(7)
    c = _ctx(4)
    W, Z, Zp = _state(c, rng)
    assert c.set_learners(2, 0.5) == 0
    for j in range(2):
        np.testing.assert_array_equal(c.replica(j), W[j])
    np.testing.assert_array_equal(c.central(), Z)
    G = rng.standard_normal((2, c.P))
    c.sma_apply(G)
    np.testing.assert_allclose(c.central(), W[:2].mean(axis=0) + 0.9 * (Z - Zp), rtol=0,
                               atol=1e-14)


def test_resizing_needs_an_iteration_barrier(oracle_lib):
    c = _ctx(2, b=2)
    x, y = wl.batch(4, 1, 28, 28, 10, 0, 0)
    c.step(x, y)
    assert c.set_learners(3, 1.0 / 3) == -4
    assert c.sync() == 0
    assert c.set_learners(3, 1.0 / 3) == 0
    assert c.set_learners(0, 1.0) == -1


def test_algorithm2_decisions(oracle_lib):
    # threshold 20 images/s; capacity 3.  Starting at one learner:
    #   t: 100 (from 0: +100 > 20 -> 2), 150 (+50 -> 3), 190 (+40, at capacity -> 3),
    #   200 (+10, not above the threshold -> 3), 170 (fell -> 2), 170 (same -> 2),
    #   160 (fell -> 1), 150 (fell, but at least one learner -> 1)
    seq = [100, 150, 190, 200, 170, 170, 160, 150]
    want = [2, 3, 3, 3, 2, 2, 1, 1]
    l, tp = 1, 0.0
    got = []
    for t in seq:
        l = oracle.tuner_next(l, t, tp, 20.0, 3)
        tp = t
        got.append(l)
    assert got == want
    # exactly at the threshold is not "above" it
    assert oracle.tuner_next(4, 120.0, 100.0, 20.0, 8) == 4
    assert oracle.tuner_next(4, 120.5, 100.0, 20.0, 8) == 5

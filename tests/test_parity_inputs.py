"""Inputs that the GPU checks rely on to take no ambiguous decision (CPU
only, oracle only).

At margin >= parity.MARGIN no fp32 rounding can flip a ReLU or max-pool
decision.  The smoke check compares three iterations without resolving
decisions, and a step whose gradient is applied as a local step (no
synchronisation in between) cannot take resolved outcomes into the
oracle's state; so those steps' inputs must have that margin, along the
oracle's own trajectory."""
import numpy as np
import pytest

import oracle
import workloads as wl
from parity import MARGIN


def f32(v):
    return float(np.float32(v))


# (what, arch, (C, H, W), classes, k, b, seed, mu, mu_l, steps, steps synced after)
CASES = [
    ("smoke", "lenet5", (1, 28, 28), 10, 2, 4, 0, 0.9, 0.0, (0, 1, 2), (0, 1, 2)),
    ("learner momentum, unsynced", "lenet5", (1, 28, 28), 10, 3, 5, 5, 0.9, 0.9, (0, 1),
     (0,)),
    ("EA-SGD, sync interval 3", "lenet5", (1, 28, 28), 10, 3, 5, 5, 0.0, 0.0, (0, 1, 3, 4),
     (2, 5)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_inputs_have_unambiguous_decisions(oracle_lib, case):
    _, arch, shape, classes, k, b, seed, mu, mu_l, check, synced = case
    m = oracle.model(arch, *shape, classes)
    w0 = wl.init_w0(oracle.tensors(m), seed)
    s = oracle.SMA(m, w0, k, b, f32(1.0 / k), f32(0.01), f32(mu), f32(mu_l))
    for t in range(max(check) + 1):
        x, y = wl.batch(k * b, *shape, classes, seed, t)
        s.step(x, y)
        if t in check:
            for j in range(k):
                margin = oracle.learner_margin(m, s.replica(j), x[j * b:(j + 1) * b],
                                               y[j * b:(j + 1) * b])
                assert margin >= MARGIN, (case[0], t, j, margin)
        if t in synced:
            assert s.sync() == 0


def test_margin_detects_a_decision_at_zero(oracle_lib):
    """A ReLU input that is exactly zero (a blank patch under a zero bias)
    gives margin 0; the same image without the patch does not."""
    m = oracle.model("lenet5", 1, 28, 28, 10)
    w = wl.init_w0(oracle.tensors(m), 0)
    x, y = wl.batch(1, 1, 28, 28, 10, seed=3)
    assert oracle.learner_margin(m, w, x, y) > 0.0
    x[:, :, 8:20, 8:20] = 0.0
    assert oracle.learner_margin(m, w, x, y) == 0.0

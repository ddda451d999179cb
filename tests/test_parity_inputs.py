"""The inputs of the strict end-to-end parity tests make every ReLU and
max-pool decision unambiguous at fp32 resolution (CPU only, oracle only).

At margin >= parity.MARGIN no fp32 rounding can flip a decision, so the
GPU tests on these inputs can hold the one-step bar exactly."""
import pytest

import oracle
import workloads as wl
from parity import MARGIN

# (arch, (C, H, W), classes, k, b, seed) of the strict end-to-end cases
STRICT = [
    ("lenet5", (1, 28, 28), 10, 2, 4, 0),
    ("lenet5", (1, 28, 28), 10, 3, 5, 5),
    ("resnet32", (3, 16, 16), 10, 2, 3, 1),
]


@pytest.mark.parametrize("arch,shape,classes,k,b,seed", STRICT)
def test_strict_inputs_have_unambiguous_decisions(oracle_lib, arch, shape, classes, k, b, seed):
    m = oracle.model(arch, *shape, classes)
    w0 = wl.init_w0(oracle.tensors(m), seed)
    x, y = wl.batch(k * b, *shape, classes, seed, 0)
    for j in range(k):
        margin = oracle.learner_margin(m, w0, x[j * b:(j + 1) * b], y[j * b:(j + 1) * b])
        assert margin >= MARGIN, (arch, j, margin)


def test_margin_detects_a_decision_at_zero(oracle_lib):
    """A ReLU input that is exactly zero (a blank patch under a zero bias)
    gives margin 0; the same image without the patch does not."""
    import numpy as np
    m = oracle.model("lenet5", 1, 28, 28, 10)
    w = wl.init_w0(oracle.tensors(m), 0)
    x, y = wl.batch(1, 1, 28, 28, 10, seed=3)
    assert oracle.learner_margin(m, w, x, y) > 0.0
    x[:, :, 8:20, 8:20] = 0.0
    assert oracle.learner_margin(m, w, x, y) == 0.0

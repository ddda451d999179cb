"""Pins for the oracle's whole-network loss and gradient (CPU only).

* Table 1 sizes: ResNet-50's parameter count times 4 bytes is the printed
  97.49 MB exactly; the input sizes match fp32 images.
* An independent float64 implementation of each declared architecture in
  torch, differentiated by autograd, must give the oracle's loss and
  gradient to rounding.
* Central finite differences of the oracle's own loss must match its
  gradient (Sec. 2.1: the gradient is that of the mean loss, Eq. 2).
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
MIB = 2.0 ** 20


def test_table1_parameter_counts(oracle_lib):
    t1 = json.load(open(os.path.join(GOLDEN, "table1.json")))
    p50 = oracle.num_params(oracle.model("resnet50", 3, 224, 224, 1000))
    assert p50 == 25_557_032
    assert round(p50 * 4 / MIB, 2) == t1["models"]["resnet50"]["model_mb"]
    p32 = oracle.num_params(oracle.model("resnet32", 3, 32, 32, 10))
    assert p32 == 464_154
    # printed 1.79 MB; option A has no shortcut weights, 1.77 MiB: within 1.2%
    assert abs(p32 * 4 / MIB - t1["models"]["resnet32"]["model_mb"]) / 1.79 < 0.012
    assert oracle.num_params(oracle.model("lenet5", 1, 28, 28, 10)) == 61_706


def test_table1_input_sizes_are_fp32():
    t1 = json.load(open(os.path.join(GOLDEN, "table1.json")))
    for name, tol in (("cifar10", 0.005), ("ilsvrc", 0.005), ("mnist", 0.01)):
        d = t1["datasets"][name]
        mb = d["images"] * int(np.prod(d["shape"])) * 4 / MIB
        assert abs(mb - d["input_mb"]) <= tol, (name, mb)


# --- an independent torch implementation of the declared architectures ----

def _params(m):
    return [(off, kind, shape) for off, kind, shape in oracle.tensors(m)]


class Cursor:
    def __init__(self, w, layout):
        self.w, self.layout, self.i = w, layout, 0

    def take(self):
        off, _, shape = self.layout[self.i]
        self.i += 1
        n = int(np.prod(shape))
        return self.w[off:off + n].view(*shape)


def torch_lenet(c, x):
    w1, b1, w2, b2 = c.take(), c.take(), c.take(), c.take()
    h = F.max_pool2d(F.relu(F.conv2d(x, w1, b1, padding=2)), 2)
    h = F.max_pool2d(F.relu(F.conv2d(h, w2, b2)), 2).flatten(1)
    for last in (False, False, True):
        W, b = c.take(), c.take()
        h = F.linear(h, W, b)
        if not last:
            h = F.relu(h)
    return h


def _cbn(c, x, st, pad):
    w = c.take()
    g, b = c.take(), c.take()
    return F.batch_norm(F.conv2d(x, w, stride=st, padding=pad), None, None, g, b, training=True,
                        eps=1e-5)


def torch_resnet32(c, x):
    h = F.relu(_cbn(c, x, 1, 1))
    cin = 16
    for stage in range(3):
        cout = 16 << stage
        for i in range(5):
            st = 2 if (stage > 0 and i == 0) else 1
            a = F.relu(_cbn(c, h, st, 1))
            bb = _cbn(c, a, 1, 1)
            sc = h[:, :, ::st, ::st]
            if cout != cin:
                sc = F.pad(sc, (0, 0, 0, 0, 0, cout - cin))
            h = F.relu(bb + sc)
            cin = cout
    h = h.mean(dim=(2, 3))
    W, b = c.take(), c.take()
    return F.linear(h, W, b)


def torch_resnet50(c, x):
    h = F.relu(_cbn(c, x, 2, 3))
    h = F.max_pool2d(h, 3, 2, 1)
    for stage, depth in enumerate((3, 4, 6, 3)):
        for i in range(depth):
            st = 2 if (stage > 0 and i == 0) else 1
            a = F.relu(_cbn(c, h, st, 0))
            a = F.relu(_cbn(c, a, 1, 1))
            a = _cbn(c, a, 1, 0)
            sc = _cbn(c, h, st, 0) if i == 0 else h
            h = F.relu(a + sc)
    h = h.mean(dim=(2, 3))
    W, b = c.take(), c.take()
    return F.linear(h, W, b)


TORCH_NETS = {"lenet5": torch_lenet, "resnet32": torch_resnet32, "resnet50": torch_resnet50}

NET_CASES = [
    ("lenet5", 1, 28, 28, 10, 3),
    ("lenet5", 2, 16, 20, 7, 2),
    ("resnet32", 3, 16, 16, 10, 2),
    ("resnet32", 3, 8, 12, 5, 3),
    ("resnet50", 3, 32, 32, 20, 4),
]


@pytest.mark.parametrize("arch,C,H,W,classes,b", NET_CASES)
def test_network_gradient_matches_torch_autograd(oracle_lib, arch, C, H, W, classes, b):
    m = oracle.model(arch, C, H, W, classes)
    layout = _params(m)
    w0 = wl.init_w0(layout, seed=7)
    rng = np.random.default_rng(11)
    # perturb BN affine params and biases away from their init so they matter
    w0 = (w0 + 0.1 * rng.standard_normal(w0.size).astype(np.float32)).astype(np.float32)
    x, y = wl.batch(b, C, H, W, classes, seed=5)
    loss, g = oracle.learner_grad(m, w0, x, y)

    wt = torch.tensor(w0.astype(np.float64), dtype=torch.float64, requires_grad=True)
    logits = TORCH_NETS[arch](Cursor(wt, layout), torch.tensor(x.astype(np.float64), dtype=torch.float64))
    lt = F.cross_entropy(logits, torch.tensor(y, dtype=torch.long))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-10 * max(1.0, abs(loss))
    gt = wt.grad.numpy()
    for off, kind, shape in layout:
        n = int(np.prod(shape))
        a, r = g[off:off + n], gt[off:off + n]
        scale = max(np.abs(r).max(), 1e-30)
        assert np.abs(a - r).max() / scale < 1e-9, (arch, off, kind, shape)


FD_CASES = [
    ("lenet5", 1, 28, 28, 10, 2),
    ("resnet32", 3, 8, 8, 10, 2),
    ("resnet50", 3, 32, 32, 10, 4),
]


@pytest.mark.parametrize("arch,C,H,W,classes,b", FD_CASES)
def test_network_gradient_finite_differences(oracle_lib, arch, C, H, W, classes, b):
    m = oracle.model(arch, C, H, W, classes)
    layout = _params(m)
    w0 = wl.init_w0(layout, seed=3).astype(np.float64)
    rng = np.random.default_rng(9)
    w0 += 0.05 * rng.standard_normal(w0.size)
    x, y = wl.batch(b, C, H, W, classes, seed=8)
    _, g = oracle.learner_grad(m, w0, x, y)
    h = 1e-7  # small enough that no ReLU or max-pool kink lies within +-h
    checked = 0
    for ti, (off, kind, shape) in enumerate(layout):
        per_tensor = 2
        if arch == "resnet50":
            if ti % 25:
                continue  # a spread of tensors keeps the test short; the
            per_tensor = 1  # autograd test above covers every tensor
        n = int(np.prod(shape))
        for e in rng.choice(n, size=min(per_tensor, n), replace=False):
            i = off + int(e)
            wp = w0.copy(); wp[i] += h
            wm = w0.copy(); wm[i] -= h
            lp, _ = oracle.learner_grad(m, wp, x, y, want_grad=False)
            lm, _ = oracle.learner_grad(m, wm, x, y, want_grad=False)
            fd = (lp - lm) / (2 * h)
            assert abs(fd - g[i]) <= 1e-6 + 1e-5 * abs(g[i]), (arch, kind, shape, i, fd, g[i])
            checked += 1
    assert checked >= 6

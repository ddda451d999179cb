"""Pins for the oracle's decision listing and its flipped-decision gradient
(CPU only), and for the parity helper that resolves ambiguous decisions.

* The listed decisions must be exactly the ReLU inputs (and max-pool
  runner-ups) of an independent torch float64 forward pass whose relative
  margin is below delta, site by site in forward order.
* The gradient with chosen decisions taken the other way must equal torch
  autograd through a ReLU / max pool whose backward is forced to the same
  outcomes.
* parity.resolve_decisions, given the oracle's gradient at weights moved
  by rounding-sized noise (a stand-in for another precision), must find
  the flipped decisions and meet 1e-4 per tensor, while a planted error of
  1e-3 in one tensor must still fail.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import workloads as wl
from parity import TOL_STEP1, resolve_decisions
from test_oracle_nets import Cursor


class Act:
    """ReLU and max pool that record their inputs per site (forward order)
    and take the listed decisions the other way in the backward pass."""

    def __init__(self, flips=()):
        self.site = 0
        self.seen = []   # (kind, tensor, extra) per site
        self.flips = {}
        for s, i, a in flips:
            self.flips.setdefault(int(s), []).append((int(i), int(a)))

    def relu(self, v):
        """A flipped decision outputs 0 for a positive input and |v| for the
        rest, and passes the gradient where that output is positive."""
        s = self.site
        self.site += 1
        self.seen.append(("relu", v.detach().clone(), None))
        y = F.relu(v).detach()
        if s in self.flips:
            flat = y.view(-1).clone()
            vf = v.detach().view(-1)
            for i, _ in self.flips[s]:
                flat[i] = 0.0 if vf[i] > 0 else (-vf[i] if -vf[i] > 0 else 2.2250738585072014e-308)
            y = flat.view_as(y)
        keep = (y > 0).double()
        return y + v * keep - (v * keep).detach()

    def maxpool(self, x, K, st, pad):
        s = self.site
        self.site += 1
        N, C, H, W = x.shape
        Ho, Wo = (H + 2 * pad - K) // st + 1, (W + 2 * pad - K) // st + 1
        xp = F.pad(x, (pad, pad, pad, pad), value=float("-inf"))
        cols = F.unfold(xp.reshape(N * C, 1, H + 2 * pad, W + 2 * pad), K, stride=st)
        # first strict maximum of the fp32-rounded values, padded cells never win
        win = torch.argmax(cols.detach().float(), dim=1)          # [N*C, L]
        self.seen.append(("pool", x.detach().clone(), (K, st, pad, win.clone())))
        if s in self.flips:
            wf = win.view(-1)
            for i, a in self.flips[s]:
                oh, ow = (i % (Ho * Wo)) // Wo, i % Wo
                ih, iw = a // W, a % W
                wf[i] = (ih - (oh * st - pad)) * K + (iw - (ow * st - pad))
        sel = torch.gather(cols, 1, win.unsqueeze(1)).squeeze(1)
        top = cols.detach().max(dim=1).values
        y = top + sel - sel.detach()
        return y.view(N, C, Ho, Wo)


def _cbn(c, x, st, pad):
    w = c.take()
    g, b = c.take(), c.take()
    return F.batch_norm(F.conv2d(x, w, stride=st, padding=pad), None, None, g, b, training=True,
                        eps=1e-5)


def t_lenet(c, x, act):
    w1, b1, w2, b2 = c.take(), c.take(), c.take(), c.take()
    h = act.maxpool(act.relu(F.conv2d(x, w1, b1, padding=2)), 2, 2, 0)
    h = act.maxpool(act.relu(F.conv2d(h, w2, b2)), 2, 2, 0).flatten(1)
    for last in (False, False, True):
        W, b = c.take(), c.take()
        h = F.linear(h, W, b)
        if not last:
            h = act.relu(h)
    return h


def t_resnet32(c, x, act):
    h = act.relu(_cbn(c, x, 1, 1))
    cin = 16
    for stage in range(3):
        cout = 16 << stage
        for i in range(5):
            st = 2 if (stage > 0 and i == 0) else 1
            a = act.relu(_cbn(c, h, st, 1))
            bb = _cbn(c, a, 1, 1)
            sc = h[:, :, ::st, ::st]
            if cout != cin:
                sc = F.pad(sc, (0, 0, 0, 0, 0, cout - cin))
            h = act.relu(bb + sc)
            cin = cout
    W, b = c.take(), c.take()
    return F.linear(h.mean(dim=(2, 3)), W, b)


def t_resnet50(c, x, act):
    h = act.maxpool(act.relu(_cbn(c, x, 2, 3)), 3, 2, 1)
    for stage, depth in enumerate((3, 4, 6, 3)):
        for i in range(depth):
            st = 2 if (stage > 0 and i == 0) else 1
            a = act.relu(_cbn(c, h, st, 0))
            a = act.relu(_cbn(c, a, 1, 1))
            a = _cbn(c, a, 1, 0)
            sc = _cbn(c, h, st, 0) if i == 0 else h
            h = act.relu(a + sc)
    W, b = c.take(), c.take()
    return F.linear(h.mean(dim=(2, 3)), W, b)


NETS = {"lenet5": t_lenet, "resnet32": t_resnet32, "resnet50": t_resnet50}
CASES = [("lenet5", 1, 28, 28, 10, 2, 0.02), ("resnet32", 3, 8, 8, 10, 2, 0.01),
         ("resnet50", 3, 32, 32, 20, 4, 0.002)]


def _setup(arch, C, H, W, classes, b, seed=4):
    m = oracle.model(arch, C, H, W, classes)
    layout = oracle.tensors(m)
    rng = np.random.default_rng(seed)
    w0 = wl.init_w0(layout, seed)
    w0 = (w0 + 0.1 * rng.standard_normal(w0.size).astype(np.float32)).astype(np.float32)
    x, y = wl.batch(b, C, H, W, classes, seed=seed + 1)
    return m, layout, w0, x, y


def _torch(arch, layout, w0, x, y, flips=()):
    wt = torch.tensor(w0.astype(np.float64), requires_grad=True)
    act = Act(flips)
    logits = NETS[arch](Cursor(wt, layout), torch.tensor(x.astype(np.float64)), act)
    loss = F.cross_entropy(logits, torch.tensor(y, dtype=torch.long))
    loss.backward()
    return loss.item(), wt.grad.numpy(), act


def _expected_decisions(act, delta):
    """The decisions within delta of turning, from torch's recorded inputs."""
    out = set()
    for s, (kind, v, extra) in enumerate(act.seen):
        rms = float(torch.sqrt((v * v).mean()))
        if kind == "relu":
            for i in torch.nonzero((v.abs() / rms).view(-1) < delta).view(-1).tolist():
                out.add((s, i, -1))
            continue
        K, st, pad, win = extra
        N, C, H, W = v.shape
        Ho, Wo = (H + 2 * pad - K) // st + 1, (W + 2 * pad - K) // st + 1
        vf = v.view(N * C, H * W)
        for nc in range(N * C):
            for o in range(Ho * Wo):
                oh, ow = o // Wo, o % Wo
                pos = int(win[nc, o])
                bh, bw = oh * st - pad + pos // K, ow * st - pad + pos % K
                best = float(vf[nc, bh * W + bw])
                if not np.float32(best) > 0:
                    continue
                for r in range(K):
                    for q in range(K):
                        ih, iw = oh * st - pad + r, ow * st - pad + q
                        if not (0 <= ih < H and 0 <= iw < W) or (ih, iw) == (bh, bw):
                            continue
                        if (best - float(vf[nc, ih * W + iw])) / rms < delta:
                            out.add((s, nc * Ho * Wo + o, ih * W + iw))
    return out


@pytest.mark.parametrize("arch,C,H,W,classes,b,delta", CASES)
def test_decisions_match_torch_forward(oracle_lib, arch, C, H, W, classes, b, delta):
    m, layout, w0, x, y = _setup(arch, C, H, W, classes, b)
    dec = oracle.learner_decisions(m, w0, x, y, delta)
    got = {(int(d["site"]), int(d["idx"]), int(d["alt"])) for d in dec}
    _, _, act = _torch(arch, layout, w0, x, y)
    want = _expected_decisions(act, delta)
    assert len(got) == len(dec)            # no decision listed twice
    assert got == want
    assert len(got) >= 3                   # the case exercises the listing
    assert np.all(dec["rel"] < delta)


@pytest.mark.parametrize("arch,C,H,W,classes,b,delta", CASES)
def test_flipped_gradient_matches_torch_autograd(oracle_lib, arch, C, H, W, classes, b, delta):
    m, layout, w0, x, y = _setup(arch, C, H, W, classes, b)
    dec = oracle.learner_decisions(m, w0, x, y, delta)
    flips = dec[::2]
    if arch != "resnet32":
        assert np.any(flips["alt"] >= 0), "the case flips a max-pool winner"
    loss, g = oracle.learner_grad_flipped(m, w0, x, y, flips)
    _, g_plain = oracle.learner_grad(m, w0, x, y)
    lt, gt, _ = _torch(arch, layout, w0, x, y,
                       [(d["site"], d["idx"], d["alt"]) for d in flips])
    assert abs(loss - lt) < 1e-10 * max(1.0, abs(loss))
    moved = 0
    for off, kind, shape in layout:
        n = int(np.prod(shape))
        a, r = g[off:off + n], gt[off:off + n]
        scale = max(np.abs(r).max(), 1e-30)
        assert np.abs(a - r).max() / scale < 1e-9, (arch, off, kind, shape)
        moved += np.abs(a - g_plain[off:off + n]).max() / scale > 1e-6
    assert moved >= 1   # the flips change the gradient


def test_resolution_finds_rounding_flips_and_rejects_real_errors(oracle_lib):
    """ResNet-32, 16 x 16 images, 8 per learner: the oracle at weights moved by
    1e-6 relative noise takes some decisions the other way (raw per-tensor
    error far above 1e-4); resolution recovers the bar with whole flips.  A
    tensor off by 1e-3, a sign flipped in one entry, or two tensors swapped
    is not absorbed."""
    m, layout, w0, x, y = _setup("resnet32", 3, 16, 16, 10, 8, seed=3)
    w = w0.astype(np.float64)
    _, g0 = oracle.learner_grad(m, w, x, y)
    wp = w * (1 + 1e-6 * np.random.default_rng(3).standard_normal(w.size))
    _, gp = oracle.learner_grad(m, wp, x, y)
    deltas = (1e-5, 3e-5)
    res = resolve_decisions(oracle, m, w, x, y, gp, layout, deltas=deltas, g0=g0)
    assert res["raw_max_rel"] > 10 * TOL_STEP1, res
    assert res["ok"] and res["flips"] >= 1 and res["err"] <= TOL_STEP1, res
    off, kind, shape = layout[20]
    n = int(np.prod(shape))
    bad = gp.copy()
    bad[off:off + n] *= 1.001
    assert not resolve_decisions(oracle, m, w, x, y, bad, layout, deltas=deltas, g0=g0)["ok"]
    bad = gp.copy()
    i = off + int(np.argmax(np.abs(g0[off:off + n])))
    bad[i] = -bad[i]
    assert not resolve_decisions(oracle, m, w, x, y, bad, layout, deltas=deltas, g0=g0)["ok"]
    bad = gp.copy()
    o2, _, s2 = layout[23]
    assert int(np.prod(s2)) == n
    bad[off:off + n], bad[o2:o2 + n] = gp[o2:o2 + n], gp[off:off + n]
    assert not resolve_decisions(oracle, m, w, x, y, bad, layout, deltas=deltas, g0=g0)["ok"]


def test_resolution_takes_duplicate_candidates_once(oracle_lib):
    """LeNet, seed 0: a conv1 ReLU input just above zero wins its 2 x 2 pooling
    window of zeros.  Taking that ReLU decision the other way, or letting any
    of the three zero cells win the window, has the same effect; a gradient
    with that effect must resolve with exactly one flip (a fit that spreads
    weight over the duplicates, or counts the effect twice, fails)."""
    m = oracle.model("lenet5", 1, 28, 28, 10)
    layout = oracle.tensors(m)
    w = wl.init_w0(layout, 0).astype(np.float64)
    x, y = wl.batch(16, 1, 28, 28, 10, 0, 0)
    dec = oracle.learner_decisions(m, w, x, y, 1e-4)
    window = dec[(dec["site"] == 1) & (dec["idx"] == 1868)]
    assert len(window) == 3
    _, g0 = oracle.learner_grad(m, w, x, y)
    _, other = oracle.learner_grad_flipped(m, w, x, y, window[:1])
    effects = [oracle.learner_grad_flipped(m, w, x, y, window[i:i + 1])[1] for i in range(3)]
    for e in effects[1:]:
        np.testing.assert_allclose(e, effects[0], rtol=0, atol=1e-15)
    res = resolve_decisions(oracle, m, w, x, y, other, layout, deltas=(1e-4,), g0=g0)
    assert res["raw_max_rel"] > 10 * TOL_STEP1, res["raw_max_rel"]
    assert res["ok"] and res["flips"] == 1, {k: v for k, v in res.items() if k != "resolved"}

"""Comparison helpers shared by the parity tests (no method arithmetic).

Bars (the method's stated tolerances): per-tensor max relative error
max|a - o| / max|o| <= 1e-4 after one step, and relative L2 of the central
model <= 1e-3 after many steps.

Decisions.  A ReLU passes its input where that input is positive, and a max
pool routes its gradient to the cell that wins its window.  When the value
a decision turns on lies within rounding of the turning point, the fp32
path and the fp64 oracle may both be right and still take it differently.
The gradients then differ by the backward effect of that one decision,
which is far above 1e-4 in the tensors below it (up to 3.5e-2 per tensor;
see resolve_decisions).  Both results are correct, so the comparison
checks that the GPU's gradient equals the oracle's gradient under *some*
valid outcome of the ambiguous decisions: the oracle lists its own
decisions within DELTA of turning (relative to the layer's RMS) and
computes the gradient with each one taken the other way; the GPU's
gradient must match the oracle's plus the effects of a subset of those
flips, each taken whole or not at all, at the stated 1e-4 per tensor.
Nothing the oracle computes depends on the GPU: the GPU's result only
selects which of the oracle's valid results it is compared with.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

TOL_STEP1 = 1e-4     # per-tensor max relative error after one step
TOL_Z_L2 = 1e-3      # relative L2 of the central model after many steps

# fp32 pre-activations deviate from fp64 by about 1e-7..1e-6 of the layer
# RMS; decisions within these relative margins are candidates, the nearer
# ones tried first.
DELTAS = (1e-6, 3e-6, 1e-5)
# Inputs whose every decision lies at least this far from turning (the
# oracle's "margin") take the same outcomes in fp32 and fp64: the smoke
# check, and the steps that an unsynchronised step follows, use such inputs.
MARGIN = 3e-6
# A candidate decision counts as taken the other way only if its whole
# effect removes more than this share of its own size from the residual.
FLIP_SLACK = 0.5


def _tensors(layout):
    for off, kind, shape in layout:
        yield off, int(np.prod(shape)), kind, shape


def tensor_errors(a, o, layout):
    """Per tensor: (max-rel, rel-L2) of a against o."""
    a = np.asarray(a, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    mr, rl = [], []
    for off, n, _, _ in _tensors(layout):
        d, r = a[off:off + n] - o[off:off + n], o[off:off + n]
        mr.append(np.abs(d).max() / max(np.abs(r).max(), 1e-30))
        rl.append(np.linalg.norm(d) / max(np.linalg.norm(r), 1e-300))
    return np.array(mr), np.array(rl)


def per_tensor_max_rel(a, o, layout):
    """max over tensors of max|a - o| / max|o| (each parameter tensor on its own)."""
    mr, _ = tensor_errors(a, o, layout)
    i = int(np.argmax(mr))
    return float(mr[i]), layout[i]


def max_rel(a, o):
    a = np.asarray(a, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    return np.abs(a - o).max() / max(np.abs(o).max(), 1e-30)


def rel_l2(a, o):
    a = np.asarray(a, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    return np.linalg.norm(a - o) / max(np.linalg.norm(o), 1e-300)


def _workers():
    return max(1, min(16, os.cpu_count() or 1))


def resolve_decisions(oracle, om, w, x, y, g, layout, tol=TOL_STEP1, deltas=DELTAS, g0=None):
    """Compares the gradient g of one learner (batch x, labels y, replica w)
    with the oracle's, resolving ambiguous decisions as described at the top.

    Returns a dict: raw_max_rel and raw_rel_l2 (the largest per-tensor errors
    before resolution), err (the largest per-tensor max-rel after), flips
    (decisions taken the other way), candidates (decisions tried), delta (the
    margin that sufficed), resolved (the oracle's gradient under the chosen
    outcomes; g0 when no flip is needed), ok."""
    if g0 is None:
        _, g0 = oracle.learner_grad(om, w, x, y)
    g = np.asarray(g, dtype=np.float64)
    raw_mr, raw_rl = tensor_errors(g, g0, layout)
    out = dict(raw_max_rel=float(raw_mr.max()), raw_rel_l2=float(raw_rl.max()), flips=0,
               candidates=0, delta=0.0, err=float(raw_mr.max()), ok=bool(raw_mr.max() <= tol),
               resolved=g0)
    if out["ok"]:
        return out
    # each tensor's rows weighted by 1 / max|o| so the fit minimises the
    # relative errors the bar is stated in
    scale = np.empty_like(g0)
    for off, n, _, _ in _tensors(layout):
        scale[off:off + n] = 1.0 / max(np.abs(g0[off:off + n]).max(), 1e-30)
    r = (g - g0) * scale
    effects, keys = [], []
    for delta in deltas:
        dec = oracle.learner_decisions(om, w, x, y, delta)
        new = [d for d in dec if (int(d["site"]), int(d["idx"]), int(d["alt"])) not in keys]
        with ThreadPoolExecutor(_workers()) as ex:
            grads = list(ex.map(lambda d: oracle.learner_grad_flipped(om, w, x, y, [d])[1], new))
        for d, gf in zip(new, grads):
            keys.append((int(d["site"]), int(d["idx"]), int(d["alt"])))
            effects.append((gf - g0) * scale)
        if not effects:
            continue
        D = np.stack(effects, axis=1)
        pick = _pick_flips(D, r)
        resolved = g0 + (D @ pick) / scale
        mr, _ = tensor_errors(g, resolved, layout)
        top = np.argsort(-mr)[:4]
        out.update(flips=int(pick.sum()), candidates=len(keys), delta=delta,
                   err=float(mr.max()), ok=bool(mr.max() <= tol), resolved=resolved,
                   worst=[(int(i), layout[i][1], tuple(layout[i][2]), float(f"{raw_mr[i]:.3g}"),
                           float(f"{mr[i]:.3g}")) for i in top])
        if out["ok"]:
            return out
    return out


def _pick_flips(D, r):
    """Whole flips (weights 0 or 1 on the columns of D) that explain r:
    repeatedly take the candidate whose whole effect shrinks the residual
    most, while one still shrinks it by more than FLIP_SLACK of that
    effect's own size.  Candidates with the same effect (a ReLU input
    within rounding of zero that wins a max-pool window of zeros appears
    as a ReLU decision and as that window's alternative winners) are taken
    once: after one of them the others would count the effect twice."""
    pick = np.zeros(D.shape[1])
    resid = r.copy()
    norms = np.einsum("ij,ij->j", D, D)
    while True:
        # |resid - D_i|^2 - |resid|^2 = |D_i|^2 - 2 <resid, D_i>
        gain = 2.0 * (resid @ D) - norms
        gain[pick > 0] = -np.inf
        i = int(np.argmax(gain))
        if not np.isfinite(gain[i]) or gain[i] <= FLIP_SLACK * norms[i]:
            return pick
        pick[i] = 1.0
        resid -= D[:, i]


def describe(tag, res, loss_err=None, margin=None):
    """One line with the achieved errors of a gradient comparison."""
    s = (f"{tag}: raw max-rel {res['raw_max_rel']:.2e} raw rel-L2 {res['raw_rel_l2']:.2e} | "
         f"resolved max-rel {res['err']:.2e} ({res['flips']} of {res['candidates']} candidate "
         f"decisions flipped, delta {res['delta']:.0e})")
    if loss_err is not None:
        s += f" | loss {loss_err:.2e}"
    if margin is not None:
        s += f" | margin {margin:.2e}"
    return s


def displacement_errors(a0, a1, r0, r1, layout, carry=None):
    """Per tensor, how far an update of the GPU's state (a0 -> a1, fp32
    values) departs from the oracle's update of the same state (r0 -> r1):
    max over elements of (|da - dr| - slack) / max|dr|, with da = a1 - a0,
    dr = r1 - r0 and slack two fp32 spacings of the larger of |a0|, |a1|
    (the GPU stores every replica and z in fp32, the oracle in fp64; an
    update of a few parts in 1e4 of a weight cannot be resolved finer than
    its storage).  Comparing displacements rather than the state itself
    keeps an update that is small next to the weights (lr = 0.01) visible at
    the 1e-4 bar.  carry (elementwise, optional) bounds how much of the
    difference comes from the start states already differing: an update
    of Algorithm 1 depends on the state through alpha (w - z) and the
    momentum terms, so states apart by rounding give updates apart by those
    coefficients times that distance."""
    a0 = np.asarray(a0, dtype=np.float32)
    a1 = np.asarray(a1, dtype=np.float32)
    da = a1.astype(np.float64) - a0.astype(np.float64)
    dr = np.asarray(r1, dtype=np.float64) - np.asarray(r0, dtype=np.float64)
    slack = 2.0 * np.spacing(np.maximum(np.abs(a0), np.abs(a1))).astype(np.float64)
    if carry is not None:
        slack = slack + carry
    excess = np.maximum(np.abs(da - dr) - slack, 0.0)
    out = []
    for off, n, _, _ in _tensors(layout):
        out.append(excess[off:off + n].max() / max(np.abs(dr[off:off + n]).max(), 1e-30))
    return np.array(out)

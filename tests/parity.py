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
# A decision counts as taken the other way when its fitted weight is
# within this distance of 1, and as not when within it of 0.
FLIP_SLACK = 0.2


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

    Returns a dict: raw (max-rel, rel-L2 per tensor before resolution),
    err (per-tensor max-rel after), flips (decisions taken the other way),
    candidates (decisions tried), delta (the margin that sufficed), ok."""
    if g0 is None:
        _, g0 = oracle.learner_grad(om, w, x, y)
    g = np.asarray(g, dtype=np.float64)
    raw_mr, raw_rl = tensor_errors(g, g0, layout)
    out = dict(raw_max_rel=float(raw_mr.max()), raw_rel_l2=float(raw_rl.max()), flips=0,
               candidates=0, delta=0.0, err=float(raw_mr.max()), ok=bool(raw_mr.max() <= tol))
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
        coef, *_ = np.linalg.lstsq(D, r, rcond=None)
        pick = np.round(np.clip(coef, 0.0, 1.0))
        resid = (r - D @ pick) / scale + g0
        mr, _ = tensor_errors(resid, g0, layout)
        whole = bool(np.all(np.abs(coef - pick) <= FLIP_SLACK))
        out.update(flips=int(pick.sum()), candidates=len(keys), delta=delta,
                   err=float(mr.max()), ok=bool(mr.max() <= tol and whole),
                   max_coef_dev=float(np.abs(coef - pick).max()))
        if out["ok"]:
            return out
    return out


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

"""Writes the stored expected values used by the GPU parity tests.

Every value here comes from the CPU oracle (``oracle/``) on the seeded
synthetic inputs of ``workloads``; nothing is read from the GPU library.
Run from the repository root:

    python tests/golden/make_golden.py lenet_envelope
    python tests/golden/make_golden.py resnet32_z100     # ~35 min single-threaded
    python tests/golden/make_golden.py resnet32_z10      # ~4 min
    python tests/golden/make_golden.py resnet32_envelope # ~1 h
    python tests/golden/make_golden.py resnet50_sampled  # ~10 min
    python tests/golden/make_golden.py lenet_z1000       # ~5 min
    python tests/golden/make_golden.py resnet50_envelope [trial]  # ~10 min per trial

Jobs:
  lenet_envelope / resnet32_envelope: how far the oracle drifts from itself
    when w0 is perturbed by one part in 1e7 (fp32 rounding level): the
    relative L2 distance of the two central models at several steps.  Any
    fp32 implementation that sums in another order can differ from the
    oracle by about this much; the long-run parity bound uses it.
  resnet32_z100 / resnet32_z10: the central model after 100 (10) SMA
    iterations of ResNet-32, k = 4 learners of batch 32 (float32 .npy).
  resnet50_sampled: learner 0's loss and sampled gradient entries after one
    forward/backward pass of ResNet-50 on 224x224 images, b = 32.
  resnet50_envelope: learner 0's gradient of the same ResNet-50 pass with w0
    perturbed by one part in 1e6 (six independent draws, one per trial
    number), at the sampled entries of resnet50_sampled: how far the
    oracle's own sampled gradient moves, per tensor, when noise of the size
    of fp32 arithmetic error flips the ReLU and max-pool decisions that lie
    within that distance of turning.  (fp32 pre-activations stray from fp64
    by up to ~1e-6..1e-5 of the layer RMS: the decisions the GPU takes the
    other way at full-size ResNet-32 lie that close to turning.)
  lenet_z1000: LeNet-5, k = 8 learners of 16, the full 1000 SMA iterations:
    the central model after 1000 (float32 .npy) and the oracle's drift
    from itself (as in the envelope jobs) after 100, 300 and 1000.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as wl  # noqa: E402

PERTURB = 1e-7
PERTURB_R50 = 1e-6
STEPS = (1, 10, 30, 50, 100)


def f32(v):
    return float(np.float32(v))


def run_sma(wk, steps, w0, keep=()):
    m = oracle.model(wk.arch, wk.in_c, wk.in_h, wk.in_w, wk.num_classes)
    s = oracle.SMA(m, w0, wk.k, wk.b, f32(wk.alpha), f32(wk.lr), f32(wk.momentum))
    kept = {}
    for t in range(steps):
        x, y = wl.workload_batch(wk, t)
        s.step(x, y)
        assert s.sync() == 0
        if t + 1 in keep:
            kept[t + 1] = s.central()
        if (t + 1) % 10 == 0 or t + 1 == steps:
            print(f"{wk.name} step {t + 1}", flush=True)
    return s, kept


def w0_of(wk, perturb=0.0):
    m = oracle.model(wk.arch, wk.in_c, wk.in_h, wk.in_w, wk.num_classes)
    w0 = wl.init_w0(oracle.tensors(m), wk.seed)
    if perturb:
        eps = np.random.default_rng(12345).standard_normal(w0.size).astype(np.float32)
        w0 = (w0 * (1 + perturb * eps)).astype(np.float32)
    return w0


def envelope(wk, out_name, steps=100):
    _, a = run_sma(wk, steps, w0_of(wk), keep=STEPS)
    _, b = run_sma(wk, steps, w0_of(wk, PERTURB), keep=STEPS)
    env = {str(t): float(np.linalg.norm(a[t] - b[t]) / np.linalg.norm(a[t])) for t in STEPS}
    doc = {"workload": wk.name, "perturbation": PERTURB,
           "what": "relative L2 distance between the oracle's central models from w0 and from "
                   "w0*(1+1e-7*N(0,1)), after each listed number of SMA iterations",
           "rel_l2": env}
    json.dump(doc, open(os.path.join(HERE, out_name), "w"), indent=1)
    print(doc)


def resnet32_z(steps):
    wk = wl.RESNET32_K4
    t0 = time.time()
    s, kept = run_sma(wk, steps, w0_of(wk), keep=(steps,))
    name = f"resnet32_k4_b32_z{steps}"
    np.save(os.path.join(HERE, name + ".npy"), kept[steps].astype(np.float32))
    json.dump({"workload": wk.name, "steps": steps, "seconds": round(time.time() - t0),
               "file": name + ".npy", "dtype": "float32 (oracle fp64 rounded)",
               "loss_last": [float(v) for v in s.loss()]},
              open(os.path.join(HERE, name + ".json"), "w"), indent=1)


def resnet50_sampled(per_tensor=24):
    wk = wl.RESNET50_K2
    m = oracle.model(wk.arch, wk.in_c, wk.in_h, wk.in_w, wk.num_classes)
    layout = oracle.tensors(m)
    w0 = w0_of(wk)
    x, y = wl.workload_batch(wk, 0)
    t0 = time.time()
    loss, g = oracle.learner_grad(m, w0, x[:wk.b], y[:wk.b])
    rng = np.random.default_rng(2024)
    entries = []
    for off, kind, shape in layout:
        n = int(np.prod(shape))
        idx = rng.choice(n, size=min(per_tensor, n), replace=False) + off
        top = off + int(np.argmax(np.abs(g[off:off + n])))
        entries.append({"offset": off, "kind": kind, "shape": list(shape),
                        "max_abs": float(np.abs(g[off:off + n]).max()),
                        "index": [int(i) for i in idx] + [top],
                        "value": [float(g[i]) for i in idx] + [float(g[top])]})
    json.dump({"workload": wk.name, "learner": 0, "b": wk.b, "loss": loss,
               "seconds": round(time.time() - t0), "tensors": entries},
              open(os.path.join(HERE, "resnet50_k2_b32_learner0.json"), "w"))


def lenet_z1000():
    wk = wl.LENET_K8
    keep = (100, 300, 1000)
    t0 = time.time()
    s, a = run_sma(wk, 1000, w0_of(wk), keep=keep)
    _, b = run_sma(wk, 1000, w0_of(wk, PERTURB), keep=keep)
    np.save(os.path.join(HERE, "lenet5_k8_b16_z1000.npy"), a[1000].astype(np.float32))
    env = {str(t): float(np.linalg.norm(a[t] - b[t]) / np.linalg.norm(a[t])) for t in keep}
    json.dump({"workload": wk.name, "steps": 1000, "file": "lenet5_k8_b16_z1000.npy",
               "dtype": "float32 (oracle fp64 rounded)", "seconds": round(time.time() - t0),
               "perturbation": PERTURB,
               "what": "relative L2 distance between the oracle's central models from w0 and from "
                       "w0*(1+1e-7*N(0,1)) after each listed number of SMA iterations",
               "rel_l2": env},
              open(os.path.join(HERE, "lenet5_k8_b16_z1000.json"), "w"), indent=1)


def resnet50_envelope(trial):
    wk = wl.RESNET50_K2
    m = oracle.model(wk.arch, wk.in_c, wk.in_h, wk.in_w, wk.num_classes)
    gold = json.load(open(os.path.join(HERE, "resnet50_k2_b32_learner0.json")))
    w0 = wl.init_w0(oracle.tensors(m), wk.seed)
    eps = np.random.default_rng(777 + trial).standard_normal(w0.size).astype(np.float32)
    w0 = (w0 * (1 + PERTURB_R50 * eps)).astype(np.float32)
    x, y = wl.workload_batch(wk, 0)
    t0 = time.time()
    loss, g = oracle.learner_grad(m, w0, x[:wk.b], y[:wk.b])
    rows = []
    for t in gold["tensors"]:
        idx = np.array(t["index"])
        d = g[idx] - np.array(t["value"])
        rows.append({"offset": t["offset"],
                     "max_rel": float(np.abs(d).max() / t["max_abs"]),
                     "rel_l2": float(np.linalg.norm(d) / max(np.linalg.norm(t["value"]), 1e-300))})
    name = f"resnet50_k2_b32_envelope{trial}.json"
    json.dump({"workload": wk.name, "learner": 0, "perturbation": PERTURB_R50, "trial": trial,
               "what": "learner 0's sampled gradient at w0*(1+1e-6*N(0,1)) against the stored "
                       "one at w0: per tensor max|d|/max|g| and relative L2 over the samples",
               "loss_rel": abs(loss - gold["loss"]) / gold["loss"],
               "seconds": round(time.time() - t0), "tensors": rows},
              open(os.path.join(HERE, name), "w"), indent=0)


if __name__ == "__main__":
    job = sys.argv[1]
    if job == "lenet_envelope":
        envelope(wl.LENET_K8, "lenet5_k8_b16_envelope.json")
    elif job == "resnet32_envelope":
        envelope(wl.RESNET32_K4, "resnet32_k4_b32_envelope.json")
    elif job == "resnet32_z100":
        resnet32_z(100)
    elif job == "resnet32_z10":
        resnet32_z(10)
    elif job == "lenet_z1000":
        lenet_z1000()
    elif job == "resnet50_envelope":
        resnet50_envelope(int(sys.argv[2]) if len(sys.argv) > 2 else 0)
    elif job == "resnet50_sampled":
        resnet50_sampled()
    else:
        raise SystemExit(f"unknown job {job}")

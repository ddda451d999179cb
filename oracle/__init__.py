"""Python access to the CPU oracle (``cbref.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  Nothing here is imported by the GPU
library or its binding, and nothing here imports them.

Every array handed back is float64.  Inputs (images, the initial model) are
passed as float32 and labels as int32, the same arrays the GPU path gets.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cbref.c")
_LIB = os.path.join(_HERE, "libcbref.so")

ARCH = {"lenet5": 1, "resnet32": 2, "resnet50": 3}
KIND_NAMES = {0: "conv_w", 1: "bias", 2: "bn_gamma", 3: "bn_beta", 4: "fc_w"}

# Built as plain ISO C, single-threaded, no contraction of a*b+c into fma and
# no fast-math, so that every rounding is the one the source spells out.
CFLAGS = ["-std=c11", "-O3", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(verbose: bool = False) -> str:
    """Compile cbref.c into libcbref.so next to it; returns the path."""
    cmd = ["gcc", *CFLAGS, _SRC, "-o", _LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class Model(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int32), ("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32),
                ("in_w", ctypes.c_int32), ("num_classes", ctypes.c_int32)]


_lib = None
_P = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        L.cbref_num_params.restype = ctypes.c_int64
        L.cbref_num_params.argtypes = [_P]
        L.cbref_num_tensors.argtypes = [_P]
        L.cbref_tensor_info.argtypes = [_P, ctypes.c_int, _P, _P, _P, _P]
        L.cbref_learner_grad.argtypes = [_P, _P, _P, _P, ctypes.c_int, _P, _P]
        L.cbref_learner_margin.argtypes = [_P, _P, _P, _P, ctypes.c_int, _P, _P]
        L.cbref_learner_decisions.argtypes = [_P, _P, _P, _P, ctypes.c_int, ctypes.c_double,
                                              ctypes.c_int, _P, _P, _P, _P, _P]
        L.cbref_learner_grad_flipped.argtypes = [_P, _P, _P, _P, ctypes.c_int, ctypes.c_int,
                                                 _P, _P, _P, _P, _P]
        L.cbref_create.restype = _P
        L.cbref_create.argtypes = [_P, _P, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                   ctypes.c_double]
        L.cbref_destroy.argtypes = [_P]
        for name in ("cbref_step",):
            getattr(L, name).argtypes = [_P, _P, _P]
        L.cbref_sync.argtypes = [_P]
        L.cbref_sma_apply.argtypes = [_P, _P]
        L.cbref_set_state.argtypes = [_P, _P, _P, _P, _P]
        L.cbref_set_lr.argtypes = [_P, ctypes.c_double]
        L.cbref_restart.argtypes = [_P]
        L.cbref_set_learners.argtypes = [_P, ctypes.c_int, ctypes.c_double]
        L.cbref_tuner_next.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double,
                                       ctypes.c_double, ctypes.c_int]
        for name in ("cbref_get_central", "cbref_get_prev_central", "cbref_get_loss"):
            getattr(L, name).argtypes = [_P, _P]
        for name in ("cbref_get_replica", "cbref_get_grad"):
            getattr(L, name).argtypes = [_P, ctypes.c_int, _P]
        L.cbref_conv2d.argtypes = [_P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                   _P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                   _P, _P, _P, _P, _P]
        L.cbref_batchnorm.argtypes = [_P, ctypes.c_int, ctypes.c_int, ctypes.c_int, _P, _P, _P,
                                      _P, _P, _P, _P]
        L.cbref_maxpool.argtypes = [_P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_int, _P, _P, _P]
        L.cbref_sma_update.argtypes = [ctypes.c_int, ctypes.c_int64, _P, _P, _P, _P, _P,
                                       ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                       ctypes.c_double, ctypes.c_int]
        L.cbref_conv_samples.argtypes = [ctypes.c_int, _P, _P, _P, _P] + [ctypes.c_int] * 8 + [
            _P, ctypes.c_int, _P]
        L.cbref_softmax_xent.restype = ctypes.c_double
        L.cbref_softmax_xent.argtypes = [_P, _P, ctypes.c_int, ctypes.c_int, _P]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def model(arch: str, in_c: int, in_h: int, in_w: int, num_classes: int) -> Model:
    return Model(ARCH[arch], in_c, in_h, in_w, num_classes)


def num_params(m: Model) -> int:
    return int(lib().cbref_num_params(ctypes.byref(m)))


def tensors(m: Model):
    """List of (offset, kind_name, shape) for every parameter tensor, in order."""
    L = lib()
    out = []
    for i in range(L.cbref_num_tensors(ctypes.byref(m))):
        off = ctypes.c_int64()
        kind = ctypes.c_int()
        nd = ctypes.c_int()
        dims = (ctypes.c_int * 4)()
        rc = L.cbref_tensor_info(ctypes.byref(m), i, ctypes.byref(off), ctypes.byref(kind),
                                 ctypes.byref(nd), dims)
        assert rc == 0
        out.append((off.value, KIND_NAMES[kind.value], tuple(dims[: nd.value])))
    return out


def learner_grad(m: Model, w, x, y, want_grad: bool = True):
    """Mean loss of one learner's batch and its gradient (Eq. 2)."""
    w = _f64(w)
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    g = np.empty_like(w) if want_grad else None
    loss = ctypes.c_double()
    rc = lib().cbref_learner_grad(ctypes.byref(m), _ptr(w), _ptr(x), _ptr(y), len(y), _ptr(g),
                                  ctypes.byref(loss))
    if rc:
        raise ValueError("cbref_learner_grad failed")
    return loss.value, g


def learner_margin(m: Model, w, x, y, with_bn=False):
    """Smallest relative distance of any ReLU input, or any max-pool winner
    from its runner-up, to the point where that decision flips (forward
    pass of one learner's batch, relative to the layer's RMS).  With
    with_bn, also the largest batch-norm conditioning factor."""
    w = _f64(w)
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    out, cond = ctypes.c_double(), ctypes.c_double()
    rc = lib().cbref_learner_margin(ctypes.byref(m), _ptr(w), _ptr(x), _ptr(y), len(y),
                                    ctypes.byref(out), ctypes.byref(cond))
    if rc:
        raise ValueError("cbref_learner_margin failed")
    return (out.value, cond.value) if with_bn else out.value


DECISION_DTYPE = np.dtype([("site", np.int32), ("idx", np.int64), ("alt", np.int64),
                           ("rel", np.float64)])


def learner_decisions(m: Model, w, x, y, delta: float):
    """Decisions of one learner's forward pass that lie within delta (relative
    to the layer's RMS) of turning the other way: a structured array with
    fields site (ReLU or max pool, numbered in forward order), idx (element
    or pooled output), alt (runner-up cell of a max-pool window, -1 for a
    ReLU) and rel (the relative margin), in forward order."""
    w = _f64(w)
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    cap = 256
    while True:
        site = np.empty(cap, np.int32)
        idx = np.empty(cap, np.int64)
        alt = np.empty(cap, np.int64)
        rel = np.empty(cap, np.float64)
        count = ctypes.c_int()
        rc = lib().cbref_learner_decisions(ctypes.byref(m), _ptr(w), _ptr(x), _ptr(y), len(y),
                                           float(delta), cap, _ptr(site), _ptr(idx), _ptr(alt),
                                           _ptr(rel), ctypes.byref(count))
        if rc:
            raise ValueError("cbref_learner_decisions failed")
        if count.value <= cap:
            break
        cap = count.value
    n = count.value
    out = np.empty(n, DECISION_DTYPE)
    out["site"], out["idx"], out["alt"], out["rel"] = site[:n], idx[:n], alt[:n], rel[:n]
    return out


def learner_grad_flipped(m: Model, w, x, y, flips):
    """Mean loss and gradient of one learner's batch with the given decisions
    (rows of learner_decisions' array) taken the other way."""
    w = _f64(w)
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    flips = np.asarray(flips, dtype=DECISION_DTYPE).reshape(-1)
    site = np.ascontiguousarray(flips["site"], dtype=np.int32)
    idx = np.ascontiguousarray(flips["idx"], dtype=np.int64)
    alt = np.ascontiguousarray(flips["alt"], dtype=np.int64)
    g = np.empty_like(w)
    loss = ctypes.c_double()
    rc = lib().cbref_learner_grad_flipped(ctypes.byref(m), _ptr(w), _ptr(x), _ptr(y), len(y),
                                          len(flips), _ptr(site), _ptr(idx), _ptr(alt), _ptr(g),
                                          ctypes.byref(loss))
    if rc:
        raise ValueError("cbref_learner_grad_flipped failed")
    return loss.value, g


class SMA:
    """Algorithm 1 on the CPU: k learners, batch b each."""

    def __init__(self, m: Model, w0, k, b, alpha, lr, momentum, learner_momentum=0.0):
        self.m = m
        self.P = num_params(m)
        w0 = np.ascontiguousarray(w0, dtype=np.float32)
        assert w0.size == self.P
        self.k, self.b = k, b
        self._c = lib().cbref_create(ctypes.byref(m), _ptr(w0), self.P, k, b, float(alpha),
                                     float(lr), float(momentum), float(learner_momentum))
        if not self._c:
            raise ValueError("cbref_create rejected the arguments")

    def __del__(self):
        if getattr(self, "_c", None):
            lib().cbref_destroy(self._c)
            self._c = None

    def step(self, x, y):
        x = np.ascontiguousarray(x, dtype=np.float32)
        y = np.ascontiguousarray(y, dtype=np.int32)
        assert len(y) == self.k * self.b
        rc = lib().cbref_step(self._c, _ptr(x), _ptr(y))
        if rc:
            raise ValueError("cbref_step failed")

    def sync(self):
        return lib().cbref_sync(self._c)

    def sma_apply(self, grads):
        g = _f64(grads).reshape(self.k, self.P)
        return lib().cbref_sma_apply(self._c, _ptr(g))

    def set_state(self, W, Z, Zp, Wprev=None):
        # every converted array is held in a local until the call returns
        W = _f64(W).reshape(self.k, self.P)
        Wp = None if Wprev is None else _f64(Wprev).reshape(self.k, self.P)
        Z, Zp = _f64(Z), _f64(Zp)
        lib().cbref_set_state(self._c, _ptr(W), _ptr(Wp), _ptr(Z), _ptr(Zp))

    def set_lr(self, lr):
        lib().cbref_set_lr(self._c, float(lr))

    def restart(self):
        lib().cbref_restart(self._c)

    def set_learners(self, k, alpha):
        rc = lib().cbref_set_learners(self._c, int(k), float(alpha))
        if rc == 0:
            self.k = int(k)
        return rc

    def central(self):
        o = np.empty(self.P)
        lib().cbref_get_central(self._c, _ptr(o))
        return o

    def prev_central(self):
        o = np.empty(self.P)
        lib().cbref_get_prev_central(self._c, _ptr(o))
        return o

    def replica(self, j):
        o = np.empty(self.P)
        assert lib().cbref_get_replica(self._c, j, _ptr(o)) == 0
        return o

    def grad(self, j):
        o = np.empty(self.P)
        assert lib().cbref_get_grad(self._c, j, _ptr(o)) == 0
        return o

    def loss(self):
        o = np.empty(self.k)
        lib().cbref_get_loss(self._c, _ptr(o))
        return o


def tuner_next(l, t, t_prev, threshold, l_max):
    """Algorithm 2, one observation (see cbref_tuner_next)."""
    return lib().cbref_tuner_next(int(l), float(t), float(t_prev), float(threshold), int(l_max))


# --- layer primitives, for pinning each against a library routine -------

def conv2d(x, w, bias, stride, pad, dy=None):
    x, w = _f64(x), _f64(w)
    N, Ci, H, W = x.shape
    Co, _, R, _ = w.shape
    Ho, Wo = (H + 2 * pad - R) // stride + 1, (W + 2 * pad - R) // stride + 1
    y = np.empty((N, Co, Ho, Wo))
    b = None if bias is None else _f64(bias)
    dx = np.empty_like(x) if dy is not None else None
    dw = np.empty_like(w) if dy is not None else None
    db = np.empty(Co) if (dy is not None and bias is not None) else None
    dyc = None if dy is None else _f64(dy)
    lib().cbref_conv2d(_ptr(x), N, Ci, H, W, _ptr(w), _ptr(b), Co, R, stride, pad, _ptr(y),
                       _ptr(dyc), _ptr(dx), _ptr(dw), _ptr(db))
    return y, dx, dw, db


def batchnorm(x, gamma, beta, dy=None):
    x = _f64(x)
    N, C = x.shape[:2]
    HW = int(np.prod(x.shape[2:]))
    y = np.empty_like(x)
    dx = np.empty_like(x) if dy is not None else None
    dg = np.empty(C) if dy is not None else None
    dbt = np.empty(C) if dy is not None else None
    dyc = None if dy is None else _f64(dy)
    gamma, beta = _f64(gamma), _f64(beta)
    lib().cbref_batchnorm(_ptr(x), N, C, HW, _ptr(gamma), _ptr(beta), _ptr(y),
                          _ptr(dyc), _ptr(dx), _ptr(dg), _ptr(dbt))
    return y, dx, dg, dbt


def maxpool(x, K, stride, pad, dy=None):
    x = _f64(x)
    N, C, H, W = x.shape
    Ho, Wo = (H + 2 * pad - K) // stride + 1, (W + 2 * pad - K) // stride + 1
    y = np.empty((N, C, Ho, Wo))
    dx = np.empty_like(x) if dy is not None else None
    dyc = None if dy is None else _f64(dy)
    lib().cbref_maxpool(_ptr(x), N, C, H, W, K, stride, pad, _ptr(y), _ptr(dyc), _ptr(dx))
    return y, dx


def softmax_xent(logits, y):
    o = _f64(logits)
    y = np.ascontiguousarray(y, dtype=np.int32)
    d = np.empty_like(o)
    loss = lib().cbref_softmax_xent(_ptr(o), _ptr(y), o.shape[0], o.shape[1], _ptr(d))
    return loss, d


def sma_update(W, G, Z, Zp, alpha, lr, mu, mu_l=0.0, Wprev=None, correct=True):
    """One synchronisation of Algorithm 1 on [k][n] replicas; returns new
    (W, Wprev, Z, Zp) as float64 arrays (inputs are not modified)."""
    W = np.array(W, dtype=np.float64, order="C")
    k = W.shape[0]
    n = W.shape[1]
    Wp = W.copy() if Wprev is None else np.array(Wprev, dtype=np.float64, order="C")
    G = _f64(G).reshape(k, n)
    Z = np.array(Z, dtype=np.float64)
    Zp = np.array(Zp, dtype=np.float64)
    lib().cbref_sma_update(k, n, _ptr(W), _ptr(Wp), _ptr(G), _ptr(Z), _ptr(Zp), float(alpha),
                           float(lr), float(mu), float(mu_l), 1 if correct else 0)
    return W, Wp, Z, Zp


def conv_samples(what, q, x=None, dy=None, w=None, bias=None, *, N, Ci, H, W, Co, R, stride, pad):
    """Conv output (what=0), weight gradient (1) or input gradient (2) at the
    index quadruples q [n, 4], each from the definition.  Arrays are fp32
    (one replica: x [N][Ci][H][W], dy [N][Co][Ho][Wo], w [Co][Ci][R][R])."""
    def f32(a):
        return None if a is None else np.ascontiguousarray(a, dtype=np.float32)
    q = np.ascontiguousarray(q, dtype=np.int32).reshape(-1, 4)
    out = np.empty(len(q))
    x, dy, w, bias = f32(x), f32(dy), f32(w), f32(bias)
    lib().cbref_conv_samples(what, _ptr(x), _ptr(dy), _ptr(w), _ptr(bias), N, Ci, H, W, Co, R,
                             stride, pad, _ptr(q), len(q), _ptr(out))
    return out

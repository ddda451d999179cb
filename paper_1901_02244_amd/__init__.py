"""MI355X library for synchronous model averaging (SMA) of k learners on one GPU.

A thin ctypes binding over ``libcrossbow_sma.so`` whose C ABI is declared in
``include/crossbow_sma.h``.  The functions keep the C names (``cb_create``,
``cb_step``, ``cb_sync``, ``cb_get_central`` ...); they only marshal
arguments.  Every step of the computation runs in the HIP kernels of the
library.  torch supplies the device memory (the workspace, images, labels)
and the stream.

Importing this package does not need a GPU; calling into the library does.
If the shared library has not been built the import of the native symbols
raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcrossbow_sma.so")

CB_OK, CB_EINVAL, CB_ENOMEM, CB_EDEVICE, CB_ESTATE, CB_ENONFINITE = 0, -1, -2, -3, -4, -5
ARCH = {"lenet5": 1, "resnet32": 2, "resnet50": 3}
KIND_NAMES = {0: "conv_w", 1: "bias", 2: "bn_gamma", 3: "bn_beta", 4: "fc_w"}

# The interface version these bindings are written for (CB_ABI_VERSION in
# include/crossbow_sma.h); a library built from other sources is refused.
ABI_VERSION = 3

# every symbol the header declares
EXPORTS = (
    "cb_abi_version", "cb_local_apply", "cb_test_conv_static", "cb_test_conv_fwd_parts", "cb_test_head_ok",
    "cb_test_head", "cb_num_params", "cb_num_tensors", "cb_tensor_info", "cb_workspace_bytes", "cb_create",
    "cb_step", "cb_sync", "cb_wait", "cb_get_central", "cb_get_replica", "cb_get_prev_central",
    "cb_get_grad", "cb_get_loss", "cb_sma_apply", "cb_set_state", "cb_last_error", "cb_destroy",
    "cb_profile_enable", "cb_profile_collect", "cb_profile_entry", "cb_profile_clear",
    "cb_test_conv_scratch_bytes", "cb_test_conv", "cb_test_bn_scratch_bytes", "cb_test_bn_fwd",
    "cb_test_bn_bwd", "cb_test_maxpool", "cb_test_softmax_xent",
    "cb_set_lr", "cb_restart", "cb_set_learners", "cb_learners", "cb_tuner_next",
    "cb_test_conv_dgrad_parts", "cb_test_conv_dgrad", "cb_set_graphs",
)


class CBError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{msg} (code {code})")
        self.code = code


class cb_model(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int32), ("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32),
                ("in_w", ctypes.c_int32), ("num_classes", ctypes.c_int32),
                ("learner_momentum", ctypes.c_float), ("check_finite", ctypes.c_int32)]


_lib = None
_P = ctypes.c_void_p


def check_abi(L, path):
    """Raises ImportError unless the loaded library L reports ABI_VERSION."""
    try:
        fn = L.cb_abi_version
    except AttributeError:
        raise ImportError(f"{path} predates interface version {ABI_VERSION} (no cb_abi_version): "
                          "rebuild it with `python -m paper_1901_02244_amd.build`") from None
    fn.restype = ctypes.c_int
    fn.argtypes = []
    v = fn()
    if v != ABI_VERSION:
        raise ImportError(f"{path} implements interface version {v}, these bindings version "
                          f"{ABI_VERSION}: rebuild it with `python -m paper_1901_02244_amd.build`")


def lib():
    """The loaded library; raises if it is missing (build it first) or was
    built from other sources than these bindings."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_1901_02244_amd.build` "
                              "(there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        check_abi(L, LIB_PATH)
        L.cb_num_params.restype = ctypes.c_int64
        L.cb_num_params.argtypes = [_P]
        L.cb_num_tensors.argtypes = [_P]
        L.cb_tensor_info.argtypes = [_P, ctypes.c_int, _P, _P, _P, _P]
        L.cb_workspace_bytes.restype = ctypes.c_size_t
        L.cb_workspace_bytes.argtypes = [_P, ctypes.c_int, ctypes.c_int]
        L.cb_create.argtypes = [_P, ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_float,
                                ctypes.c_float, _P, ctypes.c_int64, _P, ctypes.c_size_t, _P, _P]
        L.cb_step.argtypes = [_P, _P, _P]
        for n in ("cb_sync", "cb_wait"):
            getattr(L, n).argtypes = [_P]
        for n in ("cb_get_central", "cb_get_prev_central"):
            getattr(L, n).argtypes = [_P, _P, ctypes.c_int64]
        for n in ("cb_get_replica", "cb_get_grad"):
            getattr(L, n).argtypes = [_P, ctypes.c_int, _P, ctypes.c_int64]
        L.cb_get_loss.argtypes = [_P, _P]
        L.cb_sma_apply.argtypes = [_P, _P]
        L.cb_local_apply.argtypes = [_P, _P]
        L.cb_set_state.argtypes = [_P, _P, _P, _P]
        L.cb_last_error.restype = ctypes.c_char_p
        L.cb_last_error.argtypes = [_P]
        L.cb_destroy.argtypes = [_P]
        L.cb_destroy.restype = None
        L.cb_profile_enable.argtypes = [_P, ctypes.c_int]
        L.cb_profile_collect.argtypes = [_P]
        L.cb_profile_entry.argtypes = [_P, ctypes.c_int, _P, _P, _P, _P, _P]
        L.cb_profile_clear.argtypes = [_P]
        _i = ctypes.c_int
        L.cb_test_conv_scratch_bytes.restype = ctypes.c_size_t
        L.cb_test_conv_scratch_bytes.argtypes = [_i] * 9
        L.cb_test_conv_fwd_parts.argtypes = [_i] * 9
        L.cb_test_conv.argtypes = [_i] * 11 + [_P, _P, ctypes.c_int64, _P, _P, _P, _P, _P, _P,
                                               ctypes.c_size_t, _P]
        L.cb_test_conv_static.argtypes = [_i] * 11 + [_P, _P, ctypes.c_int64, _P, _P, _P, _P,
                                                      _P, _P]
        L.cb_test_head_ok.argtypes = [_i] * 4
        L.cb_test_head.argtypes = [_i] * 6 + [_P, _P, ctypes.c_int64, _P, _P, _P, _P, _P, _P, _P,
                                              _P, _i, _P, _P]
        L.cb_test_bn_scratch_bytes.restype = ctypes.c_size_t
        L.cb_test_bn_scratch_bytes.argtypes = [_i] * 5
        L.cb_test_bn_fwd.argtypes = [_i] * 6 + [_P, _P, ctypes.c_int64, _P, _P, _P, _P,
                                                ctypes.c_size_t, _P]
        L.cb_test_bn_bwd.argtypes = [_i] * 5 + [_P, _P, _i, _P, _P, ctypes.c_int64, _P, _P, _P,
                                                _P, _P, ctypes.c_size_t, _P]
        L.cb_test_maxpool.argtypes = [_i] * 7 + [_P, _P, _P, _P, _i, _P, _P]
        L.cb_test_softmax_xent.argtypes = [_i] * 3 + [_P, _P, _P, _P, _P]
        L.cb_test_conv_dgrad_parts.argtypes = [_i] * 9
        L.cb_test_conv_dgrad.argtypes = [_i] * 9 + [_P, _P, ctypes.c_int64, _P, _i, _P, _P, _i, _i,
                                                    _P, _P, _P, _P, _P, _P, _P]
        L.cb_set_lr.argtypes = [_P, ctypes.c_float]
        L.cb_restart.argtypes = [_P]
        L.cb_set_learners.argtypes = [_P, _i, ctypes.c_float]
        L.cb_learners.argtypes = [_P]
        L.cb_set_graphs.argtypes = [_P, _i]
        L.cb_tuner_next.argtypes = [_i, ctypes.c_double, ctypes.c_double, ctypes.c_double, _i]
        _lib = L
    return _lib


def model(arch: str, in_c: int, in_h: int, in_w: int, num_classes: int,
          learner_momentum: float = 0.0, check_finite: bool = False) -> cb_model:
    return cb_model(ARCH[arch], in_c, in_h, in_w, num_classes, learner_momentum,
                    1 if check_finite else 0)


def cb_num_params(m: cb_model) -> int:
    n = lib().cb_num_params(ctypes.byref(m))
    if n < 0:
        raise CBError(n, "unsupported model")
    return int(n)


def cb_tuner_next(l: int, t: float, t_prev: float, threshold: float, l_max: int) -> int:
    """Algorithm 2, one observation (the library's decision rule)."""
    return int(lib().cb_tuner_next(l, t, t_prev, threshold, l_max))


def cb_tensor_layout(m: cb_model):
    """[(offset, kind, shape)] for every parameter tensor, in order."""
    L = lib()
    out = []
    for i in range(L.cb_num_tensors(ctypes.byref(m))):
        off, kind, nd = ctypes.c_int64(), ctypes.c_int(), ctypes.c_int()
        dims = (ctypes.c_int * 4)()
        rc = L.cb_tensor_info(ctypes.byref(m), i, ctypes.byref(off), ctypes.byref(kind),
                              ctypes.byref(nd), dims)
        if rc:
            raise CBError(rc, "cb_tensor_info")
        out.append((off.value, KIND_NAMES[kind.value], tuple(dims[: nd.value])))
    return out


def cb_workspace_bytes(m: cb_model, k: int, b: int) -> int:
    return int(lib().cb_workspace_bytes(ctypes.byref(m), k, b))


def _host_f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


class Context:
    """One SMA job: k learners of batch b on the current GPU.

    The workspace is one torch uint8 tensor on the device; the stream is
    torch's current stream unless one is given."""

    def __init__(self, m: cb_model, k: int, b: int, alpha: float, lr: float, momentum: float,
                 w0, stream=None):
        import torch

        L = lib()
        self.m, self.k, self.b = m, k, b
        self.capacity = k
        self.P = cb_num_params(m)
        w0 = _host_f32(w0)
        if w0.size != self.P:
            raise CBError(CB_EINVAL, f"w0 has {w0.size} elements, the model has {self.P}")
        nbytes = cb_workspace_bytes(m, k, b)
        if nbytes == 0:
            raise CBError(CB_EINVAL, "cb_workspace_bytes rejected the model, k or b")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self._c = ctypes.c_void_p()
        rc = L.cb_create(ctypes.byref(m), k, b, alpha, lr, momentum, w0.ctypes.data, self.P,
                         self.workspace.data_ptr(), nbytes, ctypes.c_void_p(self.stream.cuda_stream),
                         ctypes.byref(self._c))
        if rc:
            raise CBError(rc, "cb_create: " + L.cb_last_error(None).decode())

    # -- errors -----------------------------------------------------------
    def _check(self, rc, what):
        if rc:
            raise CBError(rc, f"{what}: " + lib().cb_last_error(self._c).decode())
        return rc

    def close(self):
        # at interpreter exit the module globals may already be gone
        if getattr(self, "_c", None) and _lib is not None:
            _lib.cb_destroy(self._c)
        self._c = None

    __del__ = close

    # -- the method -------------------------------------------------------
    def cb_step(self, x, y):
        """x: cuda float32 [k*b][C][H][W] contiguous, y: cuda int32 [k*b]."""
        assert x.is_cuda and y.is_cuda and x.is_contiguous() and y.is_contiguous()
        assert x.dtype.is_floating_point and x.element_size() == 4 and y.element_size() == 4
        assert x.shape[0] == self.k * self.b and y.shape[0] == self.k * self.b
        assert tuple(x.shape[1:]) == (self.m.in_c, self.m.in_h, self.m.in_w)
        return self._check(lib().cb_step(self._c, x.data_ptr(), y.data_ptr()), "cb_step")

    def cb_sync(self):
        return self._check(lib().cb_sync(self._c), "cb_sync")

    def cb_wait(self):
        return self._check(lib().cb_wait(self._c), "cb_wait")

    # -- control between iterations -----------------------------------------
    def cb_set_lr(self, lr):
        return self._check(lib().cb_set_lr(self._c, lr), "cb_set_lr")

    def cb_restart(self):
        return self._check(lib().cb_restart(self._c), "cb_restart")

    def cb_set_learners(self, k, alpha):
        self._check(lib().cb_set_learners(self._c, k, alpha), "cb_set_learners")
        self.k = lib().cb_learners(self._c)
        return 0

    def cb_set_graphs(self, on=True):
        """Replay each step's launches as a HIP graph per input buffer pair."""
        return self._check(lib().cb_set_graphs(self._c, 1 if on else 0), "cb_set_graphs")

    def cb_get_central(self):
        out = np.empty(self.P, dtype=np.float32)
        self._check(lib().cb_get_central(self._c, out.ctypes.data, self.P), "cb_get_central")
        return out

    # -- test hooks -------------------------------------------------------
    def cb_get_prev_central(self):
        out = np.empty(self.P, dtype=np.float32)
        self._check(lib().cb_get_prev_central(self._c, out.ctypes.data, self.P),
                    "cb_get_prev_central")
        return out

    def cb_get_replica(self, j):
        out = np.empty(self.P, dtype=np.float32)
        self._check(lib().cb_get_replica(self._c, j, out.ctypes.data, self.P), "cb_get_replica")
        return out

    def cb_get_grad(self, j):
        out = np.empty(self.P, dtype=np.float32)
        self._check(lib().cb_get_grad(self._c, j, out.ctypes.data, self.P), "cb_get_grad")
        return out

    def cb_get_loss(self):
        out = np.empty(self.k, dtype=np.float32)
        self._check(lib().cb_get_loss(self._c, out.ctypes.data), "cb_get_loss")
        return out

    def cb_sma_apply(self, grads):
        """grads: cuda float32 [k][P] contiguous raw gradients."""
        assert grads.is_cuda and grads.is_contiguous() and grads.numel() == self.k * self.P
        return self._check(lib().cb_sma_apply(self._c, grads.data_ptr()), "cb_sma_apply")

    def cb_local_apply(self, grads):
        """A local step (no correction) with grads: cuda float32 [k][P]."""
        assert grads.is_cuda and grads.is_contiguous() and grads.numel() == self.k * self.P
        return self._check(lib().cb_local_apply(self._c, grads.data_ptr()), "cb_local_apply")

    # -- instrumentation --------------------------------------------------
    def cb_profile_enable(self, on=True):
        return self._check(lib().cb_profile_enable(self._c, 1 if on else 0), "cb_profile_enable")

    def cb_profile(self):
        """{kernel name: (launches, ms, flops, bytes)} accumulated so far."""
        L = lib()
        n = L.cb_profile_collect(self._c)
        self._check(min(n, 0), "cb_profile_collect")
        out = {}
        for i in range(n):
            name = ctypes.c_char_p()
            la, ms, fl, by = ctypes.c_int64(), ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
            self._check(L.cb_profile_entry(self._c, i, ctypes.byref(name), ctypes.byref(la),
                                           ctypes.byref(ms), ctypes.byref(fl), ctypes.byref(by)),
                        "cb_profile_entry")
            out[name.value.decode()] = (la.value, ms.value, fl.value, by.value)
        return out

    def cb_profile_clear(self):
        return self._check(lib().cb_profile_clear(self._c), "cb_profile_clear")

    def cb_set_state(self, W, z, zprev):
        W, z, zprev = _host_f32(W), _host_f32(z), _host_f32(zprev)
        assert W.size == self.k * self.P and z.size == self.P and zprev.size == self.P
        return self._check(lib().cb_set_state(self._c, W.ctypes.data, z.ctypes.data,
                                              zprev.ctypes.data), "cb_set_state")

"""The C-ABI library on the CPU: it loads, exports every declared symbol,
describes the same parameter layout as the oracle, and rejects bad
arguments before touching a device.  No compute call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_1901_02244_amd as cb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "crossbow_sma.h")

MODELS = [
    ("lenet5", 1, 28, 28, 10),
    ("lenet5", 2, 16, 20, 7),
    ("resnet32", 3, 32, 32, 10),
    ("resnet32", 3, 8, 12, 5),
    ("resnet50", 3, 224, 224, 1000),
    ("resnet50", 3, 64, 32, 20),
]


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"\b(cb_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = cb.lib()
    names = _declared()
    assert set(names) == set(cb.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("arch,C,H,W,classes", MODELS)
def test_layout_matches_oracle(oracle_lib, arch, C, H, W, classes):
    a = cb.cb_tensor_layout(cb.model(arch, C, H, W, classes))
    o = oracle.tensors(oracle.model(arch, C, H, W, classes))
    assert a == o
    assert cb.cb_num_params(cb.model(arch, C, H, W, classes)) == oracle.num_params(
        oracle.model(arch, C, H, W, classes))


def test_unsupported_models_rejected():
    for m in (cb.model("lenet5", 1, 30, 30, 10), cb.model("resnet50", 3, 48, 48, 10),
              cb.cb_model(9, 1, 28, 28, 10, 0.0, 0), cb.model("resnet32", 3, 32, 32, 0)):
        assert cb.lib().cb_num_params(ctypes.byref(m)) == cb.CB_EINVAL
        assert cb.cb_workspace_bytes(m, 2, 4) == 0
    m = cb.model("lenet5", 1, 28, 28, 10)
    assert cb.cb_workspace_bytes(m, 0, 4) == 0
    assert cb.cb_workspace_bytes(m, 2, 0) == 0


def test_workspace_grows_with_learners():
    m = cb.model("resnet32", 3, 32, 32, 10)
    sizes = [cb.cb_workspace_bytes(m, k, 16) for k in (1, 2, 4, 8, 16, 32)]
    assert all(b > a for a, b in zip(sizes, sizes[1:]))
    # replicas, gradients and activations all scale with k: roughly linear
    assert sizes[-1] < 40 * sizes[0]
    mm = cb.model("resnet32", 3, 32, 32, 10, learner_momentum=0.9)
    P = cb.cb_num_params(m)
    assert cb.cb_workspace_bytes(mm, 4, 16) - cb.cb_workspace_bytes(m, 4, 16) >= 4 * 4 * P


def test_create_validates_before_device_use():
    """Bad arguments are rejected on the host, before any HIP call."""
    L = cb.lib()
    m = cb.model("lenet5", 1, 28, 28, 10)
    P = cb.cb_num_params(m)
    w0 = np.zeros(P, dtype=np.float32)
    need = cb.cb_workspace_bytes(m, 2, 4)
    fake = ctypes.c_void_p(1 << 40)  # aligned, never dereferenced
    out = ctypes.c_void_p()

    def create(k=2, b=4, alpha=0.5, lr=0.01, mom=0.9, w=w0, n=P, ws=fake, nbytes=need):
        return L.cb_create(ctypes.byref(m), k, b, alpha, lr, mom,
                           None if w is None else w.ctypes.data, n, ws, nbytes, None,
                           ctypes.byref(out))

    assert create(nbytes=need - 1) == cb.CB_ENOMEM
    assert b"smaller" in L.cb_last_error(None)
    assert create(k=0) == cb.CB_EINVAL
    assert create(b=0) == cb.CB_EINVAL
    assert create(alpha=float("nan")) == cb.CB_EINVAL
    assert create(lr=float("inf")) == cb.CB_EINVAL
    assert create(n=P + 1) == cb.CB_EINVAL
    assert create(w=None) == cb.CB_EINVAL
    assert create(ws=ctypes.c_void_p((1 << 40) + 8)) == cb.CB_EINVAL  # misaligned
    assert out.value is None
    # calls on a NULL context are rejected
    assert L.cb_sync(None) == cb.CB_EINVAL
    assert L.cb_step(None, None, None) == cb.CB_EINVAL


def test_tuner_rule_matches_oracle(oracle_lib):
    """Algorithm 2's decision rule in the library (host code) against the
    oracle's, on random throughput sequences: integer decisions, exact."""
    import oracle
    rng = np.random.default_rng(11)
    for _ in range(200):
        l_max = int(rng.integers(1, 40))
        thr = float(rng.uniform(0, 50))
        l_lib = l_ref = int(rng.integers(1, l_max + 1))
        tp = 0.0
        for t in rng.uniform(0, 1000, 30):
            l_lib = cb.cb_tuner_next(l_lib, float(t), tp, thr, l_max)
            l_ref = oracle.tuner_next(l_ref, float(t), tp, thr, l_max)
            assert l_lib == l_ref
            assert 1 <= l_lib <= l_max
            tp = float(t)


def test_abi_version_matches_header():
    src = open(HEADER).read()
    v = int(re.search(r"#define CB_ABI_VERSION (\d+)", src).group(1))
    assert cb.ABI_VERSION == v
    L = cb.lib()
    L.cb_abi_version.restype = ctypes.c_int
    assert L.cb_abi_version() == v


def _stub(tmp_path, name, body):
    src = tmp_path / f"{name}.c"
    so = tmp_path / f"lib{name}.so"  # a distinct path each: dlopen caches by path
    src.write_text(body)
    import subprocess
    subprocess.run(["gcc", "-shared", "-fPIC", str(src), "-o", str(so)], check=True)
    return ctypes.CDLL(str(so)), str(so)


def test_stale_library_is_refused(tmp_path):
    """A library built from other sources (another interface version, or one
    from before the version call existed) raises ImportError instead of
    being called with arguments it does not take."""
    L, path = _stub(tmp_path, "older", "int cb_abi_version(void) { return %d; }\n" %
                    (cb.ABI_VERSION - 1))
    with pytest.raises(ImportError, match="interface version"):
        cb.check_abi(L, path)
    L, path = _stub(tmp_path, "unversioned", "int cb_num_params(const void* m) { return -1; }\n")
    with pytest.raises(ImportError, match="predates"):
        cb.check_abi(L, path)
    L, path = _stub(tmp_path, "current", "int cb_abi_version(void) { return %d; }\n" %
                    cb.ABI_VERSION)
    cb.check_abi(L, path)

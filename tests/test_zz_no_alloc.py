"""The entry point for callers that cannot allocate (cb_test_conv_static)
against the one with caller scratch (cb_test_conv), through the C ABI (GPU).

Both run the same kernels, so their outputs must agree bitwise: two calls
in a row, the second on a smaller layer (the library's scratch then holds
the first call's partials), and a layer whose partials exceed the
library's scratch is refused without touching its outputs."""
import zlib

import numpy as np
import pytest

import paper_1901_02244_amd as cb

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _layer(name, k, b, Ci, H, Co, R, st, pad, relu, bias):
    """Seeded inputs of one conv layer and output buffers for two runs."""
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    Ho = (H + 2 * pad - R) // st + 1
    nw = Co * Ci * R * R
    pstride = nw + (Co if bias else 0) + 3
    params = (rng.standard_normal(k * pstride) * np.sqrt(2.0 / (Ci * R * R))).astype(np.float32)
    x = rng.standard_normal((k * b, Ci, H, H), dtype=np.float32)
    dy = rng.standard_normal((k * b, Co, Ho, Ho), dtype=np.float32)
    return dict(geo=(k, b, Ci, H, H, Co, R, st, pad, relu, bias), pstride=pstride,
                x=_dev(x), p=_dev(params), dy=_dev(dy), Ho=Ho, Co=Co, Ci=Ci, k=k, b=b, H=H)


def _outputs(L):
    k, b, Co, Ho = L["k"], L["b"], L["Co"], L["Ho"]
    parts = cb.lib().cb_test_conv_fwd_parts(*L["geo"][:9])
    return dict(y=torch.full((k * b, Co, Ho, Ho), float("nan"), device="cuda"),
                stats=torch.full((k * Co * parts * 2,), float("nan"), dtype=torch.float64,
                                 device="cuda"),
                dx=torch.full_like(L["x"], float("nan")),
                g=torch.zeros_like(L["p"]))


def _run(L, static):
    lib = cb.lib()
    o = _outputs(L)
    s = torch.cuda.current_stream().cuda_stream
    args = (*L["geo"], L["x"].data_ptr(), L["p"].data_ptr(), L["pstride"], o["y"].data_ptr(),
            o["stats"].data_ptr(), L["dy"].data_ptr(), o["dx"].data_ptr(), o["g"].data_ptr())
    if static:
        rc = lib.cb_test_conv_static(*args, s)
    else:
        n = lib.cb_test_conv_scratch_bytes(*L["geo"][:9])
        scratch = torch.empty(n, dtype=torch.uint8, device="cuda")
        rc = lib.cb_test_conv(*args, scratch.data_ptr(), n, s)
    torch.cuda.synchronize()
    return rc, {k_: v.cpu().numpy() for k_, v in o.items()}


def test_static_scratch_matches_caller_scratch():
    # the largest ResNet-50 weight-gradient partials first (18 MiB), then a
    # smaller ResNet-32 layer on the scratch that still holds them
    layers = [("r50.s4.b", 2, 32, 512, 7, 512, 3, 1, 1, 0, 0),
              ("r32.s1", 4, 32, 16, 32, 16, 3, 1, 1, 0, 0)]
    need = [cb.lib().cb_test_conv_scratch_bytes(*_layer(*c)["geo"][:9]) for c in layers]
    assert need[0] > need[1] > 0 and need[0] <= 32 << 20, need
    for c in layers:
        L = _layer(*c)
        rc0, ref = _run(L, static=False)
        rc1, got = _run(L, static=True)
        assert rc0 == 0 and rc1 == 0, (c[0], rc0, rc1)
        for key in ("y", "stats", "dx", "g"):
            np.testing.assert_array_equal(got[key], ref[key], err_msg=f"{c[0]} {key}")


def test_static_scratch_refuses_larger_layers():
    c = ("r50.s4.b.k4", 4, 32, 512, 7, 512, 3, 1, 1, 0, 0)
    L = _layer(*c)
    assert cb.lib().cb_test_conv_scratch_bytes(*L["geo"][:9]) > 32 << 20
    rc, out = _run(L, static=True)
    assert rc == cb.CB_ENOMEM
    assert np.isnan(out["y"]).all() and np.isnan(out["dx"]).all()
    msg = cb.lib().cb_last_error(None).decode()
    assert "cb_test_conv_static" in msg and "bytes" in msg

"""Kernel-level parity through the operator test hooks of the C ABI (GPU).

Each operator of the learning task runs through the same launchers as
cb_step (same kernels, same tile choices) at the exact layer shapes of the
three workloads -- LeNet k=8 b=16, ResNet-32 k=4 b=32, ResNet-50 k=2 b=32
-- and at ragged shapes that leave partial tiles.  Both sides get the same
fp32 inputs, so no ReLU or max-pool decision can differ and the method's
one-step bar (per-tensor max relative error <= 1e-4) applies to every
output.  Small layers are compared whole; for large ones the oracle
computes sampled elements one by one from the definition.
"""
import zlib

import numpy as np
import pytest

import oracle
import paper_1901_02244_amd as cb
from parity import TOL_STEP1, max_rel

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# (name, k, b, Ci, H, Co, R, stride, pad, relu, bias, need_dx)
CONV = [
    # LeNet-5, 8 learners of 16 images
    ("lenet.conv1", 8, 16, 1, 28, 6, 5, 1, 2, 1, 1, 0),
    ("lenet.conv2", 8, 16, 6, 14, 16, 5, 1, 0, 1, 1, 1),
    ("lenet.fc1", 8, 16, 400, 1, 120, 1, 1, 0, 1, 1, 1),
    ("lenet.fc2", 8, 16, 120, 1, 84, 1, 1, 0, 1, 1, 1),
    ("lenet.fc3", 8, 16, 84, 1, 10, 1, 1, 0, 0, 1, 1),
    # ResNet-32, 4 learners of 32 images
    ("r32.stem", 4, 32, 3, 32, 16, 3, 1, 1, 0, 0, 0),
    ("r32.s1", 4, 32, 16, 32, 16, 3, 1, 1, 0, 0, 1),
    ("r32.s2.down", 4, 32, 16, 32, 32, 3, 2, 1, 0, 0, 1),
    ("r32.s2", 4, 32, 32, 16, 32, 3, 1, 1, 0, 0, 1),
    ("r32.s3.down", 4, 32, 32, 16, 64, 3, 2, 1, 0, 0, 1),
    ("r32.s3", 4, 32, 64, 8, 64, 3, 1, 1, 0, 0, 1),
    ("r32.fc", 4, 32, 64, 1, 10, 1, 1, 0, 0, 1, 1),
    # ResNet-50, 2 learners of 32 images (224 x 224)
    ("r50.stem", 2, 32, 3, 224, 64, 7, 2, 3, 0, 0, 0),
    ("r50.s1.a", 2, 32, 64, 56, 64, 1, 1, 0, 0, 0, 1),
    ("r50.s1.b", 2, 32, 64, 56, 64, 3, 1, 1, 0, 0, 1),
    ("r50.s1.c", 2, 32, 64, 56, 256, 1, 1, 0, 0, 0, 1),
    ("r50.s1.a2", 2, 32, 256, 56, 64, 1, 1, 0, 0, 0, 1),
    ("r50.s2.a", 2, 32, 256, 56, 128, 1, 2, 0, 0, 0, 1),
    ("r50.s2.proj", 2, 32, 256, 56, 512, 1, 2, 0, 0, 0, 1),
    ("r50.s2.b", 2, 32, 128, 28, 128, 3, 1, 1, 0, 0, 1),
    ("r50.s3.b", 2, 32, 256, 14, 256, 3, 1, 1, 0, 0, 1),
    ("r50.s3.c", 2, 32, 256, 14, 1024, 1, 1, 0, 0, 0, 1),
    ("r50.s4.a", 2, 32, 1024, 14, 512, 1, 2, 0, 0, 0, 1),
    ("r50.s4.b", 2, 32, 512, 7, 512, 3, 1, 1, 0, 0, 1),
    ("r50.s4.a2", 2, 32, 2048, 7, 512, 1, 1, 0, 0, 0, 1),
    ("r50.fc", 2, 32, 2048, 1, 1000, 1, 1, 0, 0, 1, 1),
    # 3x3 stride-1 layers of the direct kernel: every tile choice, bias and
    # ReLU, channel counts that are not multiples of 32, k = 1 and k = 32
    ("direct.w32.k1", 1, 16, 16, 32, 16, 3, 1, 1, 0, 0, 1),
    ("r32.s1.k2b16", 2, 16, 16, 32, 16, 3, 1, 1, 0, 0, 1),
    ("r32.s1.k32b16", 32, 16, 16, 32, 16, 3, 1, 1, 0, 0, 1),
    ("direct.w32.bias", 2, 3, 16, 32, 16, 3, 1, 1, 1, 1, 1),
    ("direct.w32.16to32", 2, 4, 16, 32, 32, 3, 1, 1, 1, 0, 1),
    ("direct.w16.c48", 3, 2, 48, 16, 48, 3, 1, 1, 1, 1, 1),
    ("direct.w16.k32", 32, 16, 32, 16, 32, 3, 1, 1, 0, 0, 1),
    ("direct.w8.32to64", 1, 16, 32, 8, 64, 3, 1, 1, 0, 1, 1),
    ("direct.w8.k32", 32, 16, 64, 8, 64, 3, 1, 1, 0, 0, 1),
    # 3x3 stride-2 data gradients by pixel parity
    ("s2.w32.k1", 1, 16, 16, 32, 32, 3, 2, 1, 0, 0, 1),
    ("s2.w16.c48", 3, 2, 48, 16, 32, 3, 2, 1, 1, 1, 1),
    ("s2.w16.k32", 32, 16, 32, 16, 64, 3, 2, 1, 0, 0, 1),
    # ragged: partial tiles in every GEMM dimension
    ("ragged.3x3s2", 3, 5, 7, 13, 19, 3, 2, 1, 0, 0, 1),
    ("ragged.5x5", 2, 3, 5, 11, 37, 5, 1, 2, 1, 1, 1),
    ("ragged.1x1s2", 3, 2, 70, 9, 45, 1, 2, 0, 0, 0, 1),
    ("ragged.fc", 5, 3, 33, 1, 17, 1, 1, 0, 1, 1, 1),
    # FC layers too wide for the one-wave FC kernels (the MFMA FC kernels),
    # with 1, 2 and 4 fragments of 16 images and ragged tiles
    ("ragged.fc.b9", 2, 9, 1028, 1, 264, 1, 1, 0, 0, 1, 1),
    ("ragged.fc.wide", 3, 21, 1100, 1, 300, 1, 1, 0, 1, 1, 1),
    ("ragged.fc.b50", 2, 50, 1040, 1, 260, 1, 1, 0, 0, 0, 1),
    ("ragged.7x7s2", 2, 3, 3, 19, 5, 7, 2, 3, 0, 0, 0),
    # ragged again with channel counts that take the tap-major GEMM loaders
    # (channels a multiple of the stage depth), incl. the grid-only stride-2
    # data gradient with and without its float4 epilogue
    ("ragged.tap3x3", 3, 5, 32, 13, 48, 3, 1, 1, 1, 1, 1),
    ("ragged.tap1x1", 2, 7, 64, 9, 80, 1, 1, 0, 0, 0, 1),
    ("ragged.tap1x1s2", 2, 3, 64, 10, 96, 1, 2, 0, 0, 0, 1),
    ("ragged.tap1x1s2v", 2, 3, 32, 16, 64, 1, 2, 0, 0, 0, 1),
]

FULL_LIMIT = 6e8  # multiply-adds per replica below which the oracle does whole tensors


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _rng(tag):
    return np.random.default_rng(zlib.crc32(tag.encode()))


def _sample_idx(rng, shape, n):
    return np.stack([rng.integers(0, d, n) for d in shape], axis=1).astype(np.int32)


@pytest.mark.parametrize("case", CONV, ids=[c[0] for c in CONV])
def test_conv_kernels(case):
    name, k, b, Ci, H, Co, R, st, pad, relu, bias, need_dx = case
    W = H
    Ho = (H + 2 * pad - R) // st + 1
    rng = _rng("conv" + name)
    nw = Co * Ci * R * R
    pstride = nw + (Co if bias else 0) + 3  # an odd stride between replicas
    x = rng.standard_normal((k * b, Ci, H, W), dtype=np.float32)
    params = np.zeros(k * pstride, dtype=np.float32)
    for j in range(k):
        params[j * pstride:j * pstride + nw] = rng.standard_normal(nw) * np.sqrt(2.0 / (Ci * R * R))
        if bias:
            params[j * pstride + nw:j * pstride + nw + Co] = rng.standard_normal(Co) * 0.1
    dy = rng.standard_normal((k * b, Co, Ho, Ho), dtype=np.float32)
    L = cb.lib()
    scratch_n = L.cb_test_conv_scratch_bytes(k, b, Ci, H, W, Co, R, st, pad)
    assert scratch_n > 0
    # the batch-norm statistics epilogue of every conv that is not an FC layer
    # (an FC layer with statistics would leave the FC kernel)
    parts = L.cb_test_conv_fwd_parts(k, b, Ci, H, W, Co, R, st, pad) if H > 1 else 0
    xd, pd, dyd = _dev(x), _dev(params), _dev(dy)
    yd = torch.empty((k * b, Co, Ho, Ho), dtype=torch.float32, device="cuda")
    dxd = torch.empty_like(xd) if need_dx else None
    gd = torch.zeros_like(pd)
    scratch = torch.empty(scratch_n, dtype=torch.uint8, device="cuda")
    stats = torch.full((max(1, k * Co * parts * 2),), float("nan"), dtype=torch.float64,
                       device="cuda")
    rc = L.cb_test_conv(k, b, Ci, H, W, Co, R, st, pad, relu, bias, xd.data_ptr(), pd.data_ptr(),
                        pstride, yd.data_ptr(), stats.data_ptr() if parts else None, dyd.data_ptr(),
                        dxd.data_ptr() if need_dx else None, gd.data_ptr(), scratch.data_ptr(),
                        scratch_n, torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    y, g = yd.cpu().numpy(), gd.cpu().numpy()
    dx = dxd.cpu().numpy() if need_dx else None
    # the statistics epilogue: per replica and channel the sums over the
    # replica's b images of the stored y and of y*y
    sums = stats.cpu().numpy().reshape(k, Co, parts, 2).sum(axis=2) if parts else None
    macs = b * Ho * Ho * Co * Ci * R * R
    geo = dict(N=b, Ci=Ci, H=H, W=W, Co=Co, R=R, stride=st, pad=pad)
    if parts and macs > FULL_LIMIT:
        # too large for the oracle's whole output: the sums must equal those
        # of the stored y, which is compared with the oracle on samples below
        yr = y.reshape(k, b, Co, -1).astype(np.float64)
        assert max_rel(sums[..., 0], yr.sum(axis=(1, 3))) <= TOL_STEP1, (name, "sum y")
        assert max_rel(sums[..., 1], (yr * yr).sum(axis=(1, 3))) <= TOL_STEP1, (name, "sum y*y")
    for j in range(k):
        sl = slice(j * b, (j + 1) * b)
        w = params[j * pstride:j * pstride + nw].reshape(Co, Ci, R, R)
        bb = params[j * pstride + nw:j * pstride + nw + Co] if bias else None
        gw = g[j * pstride:j * pstride + nw].reshape(Co, Ci, R, R)
        if macs <= FULL_LIMIT:
            yo, dxo, dwo, dbo = oracle.conv2d(x[sl], w, bb, st, pad, dy=dy[sl])
            if relu:
                yo = np.maximum(yo, 0.0)
            assert max_rel(y[sl], yo) <= TOL_STEP1, (name, j, "y")
            if parts:
                assert max_rel(sums[j, :, 0], yo.sum(axis=(0, 2, 3))) <= TOL_STEP1, (name, j, "sum y")
                assert max_rel(sums[j, :, 1], (yo * yo).sum(axis=(0, 2, 3))) <= TOL_STEP1, \
                    (name, j, "sum y*y")
            assert max_rel(gw, dwo) <= TOL_STEP1, (name, j, "dw")
            if bias:
                assert max_rel(g[j * pstride + nw:j * pstride + nw + Co], dbo) <= TOL_STEP1
            if need_dx:
                assert max_rel(dx[sl], dxo) <= TOL_STEP1, (name, j, "dx")
        else:
            qy = _sample_idx(rng, (b, Co, Ho, Ho), 512)
            yo = oracle.conv_samples(0, qy, x=x[sl], w=w, bias=bb, **geo)
            if relu:
                yo = np.maximum(yo, 0.0)
            ys = y[sl][tuple(qy.T)]
            assert max_rel(ys, yo) <= TOL_STEP1, (name, j, "y")
            qw = _sample_idx(rng, (Co, Ci, R, R), 256)
            assert max_rel(gw[tuple(qw.T)], oracle.conv_samples(1, qw, x=x[sl], dy=dy[sl], **geo)) \
                <= TOL_STEP1, (name, j, "dw")
            if need_dx:
                qx = _sample_idx(rng, (b, Ci, H, W), 512)
                assert max_rel(dx[sl][tuple(qx.T)],
                               oracle.conv_samples(2, qx, dy=dy[sl], w=w, **geo)) <= TOL_STEP1, \
                    (name, j, "dx")


# (name, k, b, C, H, relu)
BN = [
    ("r32.s1", 4, 32, 16, 32, 1),
    ("r32.s2", 4, 32, 32, 16, 0),
    ("r32.s3", 4, 32, 64, 8, 1),
    ("r50.stem", 2, 32, 64, 112, 1),
    ("r50.s1.c", 2, 32, 256, 56, 0),
    ("r50.s3", 2, 32, 256, 14, 1),
    ("r50.s4.c", 2, 32, 2048, 7, 0),
    ("ragged", 3, 5, 7, 9, 1),
    ("ragged.1x1", 2, 3, 5, 1, 0),
]


@pytest.mark.parametrize("case", BN, ids=[c[0] for c in BN])
def test_batchnorm_kernels(case):
    name, k, b, C, H, relu = case
    W = H
    rng = _rng("bn" + name)
    x = (rng.standard_normal((k * b, C, H, W), dtype=np.float32) * 2 + 0.5).astype(np.float32)
    dy = rng.standard_normal((k * b, C, H, W), dtype=np.float32)
    pstride = 2 * C + 1
    params = np.zeros(k * pstride, dtype=np.float32)
    for j in range(k):
        params[j * pstride:j * pstride + C] = 1 + 0.2 * rng.standard_normal(C)
        params[j * pstride + C:j * pstride + 2 * C] = 0.2 * rng.standard_normal(C)
    gam = [params[j * pstride:j * pstride + C] for j in range(k)]
    bet = [params[j * pstride + C:j * pstride + 2 * C] for j in range(k)]
    yo = np.concatenate([oracle.batchnorm(x[j * b:(j + 1) * b], gam[j], bet[j])[0]
                         for j in range(k)])
    dyo = dy
    if relu:
        yo = np.maximum(yo, 0.0)
        # the gradient through the ReLU takes the oracle's decisions on both
        # sides (the mask is handed to the GPU kernel as an input)
        dyo = np.where(yo > 0, dy, 0.0)
    ref = [oracle.batchnorm(x[j * b:(j + 1) * b], gam[j], bet[j], dy=dyo[j * b:(j + 1) * b])
           for j in range(k)]
    L = cb.lib()
    sn = L.cb_test_bn_scratch_bytes(k, b, C, H, W)
    xd, dyd, pd = _dev(x), _dev(dy), _dev(params)
    yd = torch.empty_like(xd)
    mean = torch.empty(k * C, dtype=torch.float32, device="cuda")
    istd = torch.empty(k * C, dtype=torch.float32, device="cuda")
    scratch = torch.empty(sn, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    assert L.cb_test_bn_fwd(k, b, C, H, W, relu, xd.data_ptr(), pd.data_ptr(), pstride,
                            yd.data_ptr(), mean.data_ptr(), istd.data_ptr(), scratch.data_ptr(),
                            sn, st) == 0
    mask = _dev(yo.astype(np.float32)) if relu else None
    dxd = torch.empty_like(xd)
    gd = torch.zeros_like(pd)
    assert L.cb_test_bn_bwd(k, b, C, H, W, xd.data_ptr(), mask.data_ptr() if relu else None, 0,
                            dyd.data_ptr(), pd.data_ptr(), pstride, mean.data_ptr(),
                            istd.data_ptr(), dxd.data_ptr(), gd.data_ptr(), scratch.data_ptr(), sn,
                            st) == 0
    torch.cuda.synchronize()
    assert max_rel(yd.cpu().numpy(), yo) <= TOL_STEP1
    mu = x.reshape(k, b, C, -1).astype(np.float64).mean(axis=(1, 3))
    var = x.reshape(k, b, C, -1).astype(np.float64).var(axis=(1, 3))
    assert max_rel(mean.cpu().numpy(), mu.reshape(-1)) <= TOL_STEP1
    assert max_rel(istd.cpu().numpy(), (1 / np.sqrt(var + 1e-5)).reshape(-1)) <= TOL_STEP1
    dx = dxd.cpu().numpy()
    g = gd.cpu().numpy()
    for j in range(k):
        _, dxo, dgo, dbo = ref[j]
        assert max_rel(dx[j * b:(j + 1) * b], dxo) <= TOL_STEP1, (name, j, "dx")
        assert max_rel(g[j * pstride:j * pstride + C], dgo) <= TOL_STEP1, (name, j, "dgamma")
        assert max_rel(g[j * pstride + C:j * pstride + 2 * C], dbo) <= TOL_STEP1, (name, j, "dbeta")


def _bn_relu_from_x(x, mean, istd, gam, bet):
    """The norm's ReLU decision as the kernels take it: (x - mean) * istd in
    fp32, then gamma * t + beta rounded once (a fused multiply-add; the
    product of two fp32 values is exact in fp64), positive or not."""
    t = (x - mean[None, :, None, None]) * istd[None, :, None, None]
    v = gam[None, :, None, None].astype(np.float64) * t.astype(np.float64) + \
        bet[None, :, None, None].astype(np.float64)
    return v > 0


@pytest.mark.parametrize("case", [c for c in BN if c[-1]], ids=[c[0] for c in BN if c[-1]])
def test_batchnorm_backward_relu_mask_from_x(case):
    """A norm with a ReLU and no residual input: the backward recomputes the
    ReLU decision from x and takes exactly the forward's (checked bitwise
    against the forward's output), and its gradients match the oracle's
    given that decision."""
    name, k, b, C, H, _ = case
    W = H
    rng = _rng("bnx" + name)
    x = (rng.standard_normal((k * b, C, H, W), dtype=np.float32) * 2 + 0.5).astype(np.float32)
    dy = rng.standard_normal((k * b, C, H, W), dtype=np.float32)
    pstride = 2 * C + 1
    params = np.zeros(k * pstride, dtype=np.float32)
    for j in range(k):
        params[j * pstride:j * pstride + C] = 1 + 0.2 * rng.standard_normal(C)
        params[j * pstride + C:j * pstride + 2 * C] = 0.2 * rng.standard_normal(C)
    L = cb.lib()
    sn = L.cb_test_bn_scratch_bytes(k, b, C, H, W)
    xd, dyd, pd = _dev(x), _dev(dy), _dev(params)
    yd = torch.empty_like(xd)
    mean = torch.empty(k * C, dtype=torch.float32, device="cuda")
    istd = torch.empty(k * C, dtype=torch.float32, device="cuda")
    scratch = torch.empty(sn, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    assert L.cb_test_bn_fwd(k, b, C, H, W, 1, xd.data_ptr(), pd.data_ptr(), pstride,
                            yd.data_ptr(), mean.data_ptr(), istd.data_ptr(), scratch.data_ptr(),
                            sn, st) == 0
    dxd = torch.empty_like(xd)
    gd = torch.zeros_like(pd)
    assert L.cb_test_bn_bwd(k, b, C, H, W, xd.data_ptr(), None, 1, dyd.data_ptr(), pd.data_ptr(),
                            pstride, mean.data_ptr(), istd.data_ptr(), dxd.data_ptr(),
                            gd.data_ptr(), scratch.data_ptr(), sn, st) == 0
    torch.cuda.synchronize()
    y = yd.cpu().numpy()
    mf, isf = mean.cpu().numpy().reshape(k, C), istd.cpu().numpy().reshape(k, C)
    dx, g = dxd.cpu().numpy(), gd.cpu().numpy()
    for j in range(k):
        sl = slice(j * b, (j + 1) * b)
        gam = params[j * pstride:j * pstride + C]
        bet = params[j * pstride + C:j * pstride + 2 * C]
        on = _bn_relu_from_x(x[sl], mf[j], isf[j], gam, bet)
        np.testing.assert_array_equal(on, y[sl] > 0, err_msg=f"{name} replica {j}")
        _, dxo, dgo, dbo = oracle.batchnorm(x[sl], gam, bet, dy=np.where(on, dy[sl], 0.0))
        assert max_rel(dx[sl], dxo) <= TOL_STEP1, (name, j, "dx")
        assert max_rel(g[j * pstride:j * pstride + C], dgo) <= TOL_STEP1, (name, j, "dgamma")
        assert max_rel(g[j * pstride + C:j * pstride + 2 * C], dbo) <= TOL_STEP1, (name, j, "dbeta")


# (name, N, C, H, W, K, stride, pad, mask_relu)
POOL = [
    ("lenet.pool1", 128, 6, 28, 28, 2, 2, 0, 1),
    ("lenet.pool2", 128, 16, 10, 10, 2, 2, 0, 1),
    ("r50.pool", 64, 64, 112, 112, 3, 2, 1, 0),
    ("ragged", 3, 5, 11, 11, 3, 2, 1, 1),
    # rows too wide for the LDS tiles: the forward falls back to one thread
    # per window; the backward takes one input row per tile ...
    ("wide.rows1", 1, 2, 9, 1400, 3, 2, 1, 0),
    # ... or, wider still, falls back to one thread per input cell
    ("wide.fallback", 1, 2, 6, 4200, 3, 2, 1, 1),
]


@pytest.mark.parametrize("case", POOL, ids=[c[0] for c in POOL])
def test_maxpool_kernels(case):
    name, N, C, H, W, K, st, pad, mask = case
    rng = _rng("pool" + name)
    x = rng.standard_normal((N, C, H, W), dtype=np.float32)
    if mask:
        x = np.maximum(x, 0)  # a ReLU output, with its many zero ties
    Ho, Wo = (H + 2 * pad - K) // st + 1, (W + 2 * pad - K) // st + 1
    dy = rng.standard_normal((N, C, Ho, Wo), dtype=np.float32)
    yo, dxo = oracle.maxpool(x, K, st, pad, dy=dy)
    if mask:
        dxo = np.where(x > 0, dxo, 0.0)
    xd, dyd = _dev(x), _dev(dy)
    yd = torch.empty((N, C, Ho, Wo), dtype=torch.float32, device="cuda")
    dxd = torch.empty_like(xd)
    arg = torch.empty((N, C, Ho, Wo), dtype=torch.int32, device="cuda")
    assert cb.lib().cb_test_maxpool(N, C, H, W, K, st, pad, xd.data_ptr(), yd.data_ptr(),
                                    dyd.data_ptr(), dxd.data_ptr(), mask, arg.data_ptr(),
                                    torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(yd.cpu().numpy(), yo.astype(np.float32))
    assert max_rel(dxd.cpu().numpy(), dxo) <= 1e-6


# (name, k, b, classes)
XENT = [("lenet", 8, 16, 10), ("r32", 4, 32, 10), ("r50", 2, 32, 1000), ("ragged", 3, 5, 7),
        # a row per thread up to 32 classes, in several passes beyond 256 rows; a wave per row above
        ("rows.b300", 2, 300, 10), ("rows.c32", 3, 7, 32), ("waves.c33", 2, 5, 33),
        # beyond 1024 classes a row is read again in each pass instead of kept in registers
        ("waves.c1100", 2, 37, 1100)]


@pytest.mark.parametrize("case", XENT, ids=[c[0] for c in XENT])
def test_softmax_xent_kernel(case):
    name, k, b, classes = case
    rng = _rng("xent" + name)
    o = (rng.standard_normal((k * b, classes)) * 3).astype(np.float32)
    y = rng.integers(0, classes, k * b).astype(np.int32)
    od, yd = _dev(o), _dev(y)
    dd = torch.empty_like(od)
    ld = torch.empty(k, dtype=torch.float32, device="cuda")
    assert cb.lib().cb_test_softmax_xent(k, b, classes, od.data_ptr(), yd.data_ptr(),
                                         dd.data_ptr(), ld.data_ptr(),
                                         torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    d = dd.cpu().numpy()
    loss = ld.cpu().numpy()
    for j in range(k):
        lo, do = oracle.softmax_xent(o[j * b:(j + 1) * b], y[j * b:(j + 1) * b])
        assert abs(loss[j] - lo) / abs(lo) <= TOL_STEP1
        assert max_rel(d[j * b:(j + 1) * b], do) <= TOL_STEP1


# (name, k, b, C, H, classes, bn_relu): the ResNet-32 head at the two step
# sizes of its workloads, and a ragged one
HEAD = [("r32.k4b32", 4, 32, 64, 8, 10, 1), ("r32.k32b16", 32, 16, 64, 8, 10, 1),
        ("ragged", 3, 5, 24, 4, 7, 0), ("no_bn", 2, 3, 16, 8, 5, -1)]


@pytest.mark.parametrize("case", HEAD, ids=[c[0] for c in HEAD])
def test_fused_head_kernel(case):
    """Global average pool, FC, softmax cross-entropy and their backward down
    to the pooled tensor -- with the backward sums of the batch norm that
    produced it -- in the one launch cb_step makes, against the oracle's FC
    (a 1x1 convolution on a 1x1 image) and softmax cross-entropy, with the
    pool's mean and the norm's masks and sums written out in numpy."""
    name, k, b, C, H, classes, bn_relu = case
    HW = H * H
    L = cb.lib()
    assert L.cb_test_head_ok(C, H, H, classes) == 1
    rng = _rng("head" + name)
    N = k * b
    bn_x = rng.standard_normal((N, C, H, H), dtype=np.float32)
    mean = (rng.standard_normal((k, C)) * 0.1).astype(np.float32)
    istd = rng.uniform(0.5, 2.0, (k, C)).astype(np.float32)
    y = rng.standard_normal((N, C, H, H), dtype=np.float32)
    if bn_relu == 1:
        y = np.maximum(y, 0.0)
    pstride = classes * C + classes + 3
    params = np.zeros(k * pstride, dtype=np.float32)
    for j in range(k):
        params[j * pstride:j * pstride + classes * C] = rng.standard_normal(classes * C) / np.sqrt(C)
        params[j * pstride + classes * C:j * pstride + classes * C + classes] = \
            rng.standard_normal(classes) * 0.1
    labels = rng.integers(0, classes, N).astype(np.int32)
    use_bn = bn_relu >= 0
    d = {n_: _dev(v) for n_, v in dict(y=y, p=params, l=labels, x=bn_x, m=mean, i=istd).items()}
    feat = torch.empty((N, C), dtype=torch.float32, device="cuda")
    dlog = torch.empty((N, classes), dtype=torch.float32, device="cuda")
    loss = torch.empty(N, dtype=torch.float32, device="cuda")
    dy = torch.empty((N, C, H, H), dtype=torch.float32, device="cuda")
    part = torch.full((k * C * b * 2,), float("nan"), dtype=torch.float64, device="cuda")
    rc = L.cb_test_head(k, b, C, H, H, classes, d["y"].data_ptr(), d["p"].data_ptr(), pstride,
                        d["l"].data_ptr(), feat.data_ptr(), dlog.data_ptr(), loss.data_ptr(),
                        dy.data_ptr(), d["x"].data_ptr(), d["m"].data_ptr(), d["i"].data_ptr(),
                        max(bn_relu, 0), part.data_ptr() if use_bn else None,
                        torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    feat, dlog, loss, dy = (t.cpu().numpy() for t in (feat, dlog, loss, dy))
    sums = part.cpu().numpy().reshape(k, C, b, 2)
    for j in range(k):
        sl = slice(j * b, (j + 1) * b)
        w = params[j * pstride:j * pstride + classes * C].reshape(classes, C, 1, 1)
        bias = params[j * pstride + classes * C:j * pstride + classes * C + classes]
        g = y[sl].astype(np.float64).mean(axis=(2, 3))
        assert max_rel(feat[sl], g) <= TOL_STEP1, (name, j, "features")
        logits, _, _, _ = oracle.conv2d(g[:, :, None, None], w, bias, 1, 0)
        lo, dlo = oracle.softmax_xent(logits[:, :, 0, 0], labels[sl])
        per_image = [oracle.softmax_xent(logits[i:i + 1, :, 0, 0], labels[sl][i:i + 1])[0]
                     for i in range(b)]
        assert max_rel(loss[sl], per_image) <= TOL_STEP1, (name, j, "loss terms")
        assert abs(loss[sl].astype(np.float64).mean() - lo) / abs(lo) <= TOL_STEP1
        assert max_rel(dlog[sl], dlo) <= TOL_STEP1, (name, j, "dlogits")
        _, dg, _, _ = oracle.conv2d(g[:, :, None, None], w, bias, 1, 0,
                                    dy=dlo[:, :, None, None])
        dyo = np.broadcast_to(dg / HW, (b, C, H, H))
        assert max_rel(dy[sl], dyo) <= TOL_STEP1, (name, j, "dy")
        if use_bn:
            dd = np.where(y[sl] > 0, dyo, 0.0) if bn_relu else dyo
            xh = (bn_x[sl].astype(np.float64) - mean[j][None, :, None, None]) * \
                istd[j][None, :, None, None]
            assert max_rel(sums[j, :, :, 0].T, dd.sum(axis=(2, 3))) <= TOL_STEP1, (name, j, "sum d")
            assert max_rel(sums[j, :, :, 1].T, (dd * xh).sum(axis=(2, 3))) <= TOL_STEP1, \
                (name, j, "sum d*xh")


# (name, k, b, Ci, H, Co, R, stride, pad, accumulate, mask, add_mode, add_C, bn, bn_y:
#  0 none, 1 a y tensor, 2 a y tensor that gamma and beta recompute from bn_x,
#  3 no y: the mask is the norm's own ReLU output, recomputed from bn_x by the
#  direct stride-1 kernels and read by the others)
DGRAD_EPILOGUE = [
    ("direct.w32.same.bn", 2, 4, 16, 32, 16, 3, 1, 1, 1, 1, 1, 16, 1, 1),
    ("direct.w16.bn", 2, 3, 32, 16, 32, 3, 1, 1, 0, 0, 0, 0, 1, 1),
    ("direct.w8.acc.mask", 2, 4, 64, 8, 64, 3, 1, 1, 1, 1, 1, 64, 1, 0),
    ("s2.w32.sub.bn", 2, 4, 16, 32, 32, 3, 2, 1, 0, 0, 2, 32, 1, 1),
    ("s2.w16.acc.mask.sub.bn", 2, 4, 32, 16, 64, 3, 2, 1, 1, 1, 2, 64, 1, 0),
    ("s2.w16.same", 1, 3, 16, 16, 32, 3, 2, 1, 0, 1, 1, 16, 0, 0),
    ("gemm.3x3s2.ragged.sub.bn", 2, 3, 7, 13, 19, 3, 2, 1, 1, 1, 2, 19, 1, 1),
    ("gemm.5x5.mask", 2, 4, 6, 14, 16, 5, 1, 0, 0, 1, 0, 0, 1, 1),
    # 1x1 stride 2 on even planes: the GEMM over the output grid only
    ("gemm.1x1s2.grid.acc.mask.same.bn", 2, 3, 24, 14, 40, 1, 2, 0, 1, 1, 1, 24, 1, 1),
    ("gemm.1x1s2.grid.sub.bn", 2, 5, 20, 10, 36, 1, 2, 0, 0, 0, 2, 20, 1, 0),
    # bn_y = 2: the norm's ReLU output recomputed from bn_x (a norm with no residual input)
    ("direct.w32.same.bn.relux", 2, 4, 16, 32, 16, 3, 1, 1, 1, 0, 1, 16, 1, 2),
    ("direct.w8.bn.relux", 2, 3, 64, 8, 64, 3, 1, 1, 0, 0, 0, 0, 1, 2),
    ("s2.w16.sub.bn.relux", 2, 4, 32, 16, 64, 3, 2, 1, 0, 0, 2, 64, 1, 2),
    ("gemm.3x3s2.ragged.bn.relux", 2, 3, 7, 13, 19, 3, 2, 1, 0, 0, 0, 0, 1, 2),
    ("gemm.5x5.bn.relux", 2, 4, 6, 14, 16, 5, 1, 0, 0, 0, 0, 0, 1, 2),
    ("gemm.1x1s2.grid.acc.same.bn.relux", 2, 3, 24, 14, 40, 1, 2, 0, 1, 0, 1, 24, 1, 2),
    ("direct.w32.mask.bn.rc", 2, 4, 16, 32, 16, 3, 1, 1, 0, 1, 0, 0, 1, 3),
    ("direct.w16.acc.mask.same.bn.rc", 2, 3, 32, 16, 32, 3, 1, 1, 1, 1, 1, 32, 1, 3),
    ("direct.w8.mask.bn.rc", 2, 3, 64, 8, 64, 3, 1, 1, 0, 1, 0, 0, 1, 3),
    ("s2.w16.mask.bn.rc", 2, 4, 32, 16, 64, 3, 2, 1, 0, 1, 0, 0, 1, 3),
    ("gemm.5x5.mask.bn.rc", 2, 4, 6, 14, 16, 5, 1, 0, 0, 1, 0, 0, 1, 3),
    # the tap-major GEMM loaders (output channels a multiple of the stage
    # depth) under the full epilogue, and the grid-only stride-2 form with
    # four grid points to a grid row (its float4 epilogue)
    ("gemm.tap3x3.acc.mask.same.bn", 2, 3, 24, 13, 32, 3, 1, 1, 1, 1, 1, 24, 1, 1),
    ("gemm.tap1x1.acc.mask.same.bn.rc", 2, 3, 24, 9, 64, 1, 1, 0, 1, 1, 1, 24, 1, 3),
    ("gemm.1x1s2.grid4.acc.mask.same.bn", 2, 3, 24, 16, 64, 1, 2, 0, 1, 1, 1, 24, 1, 1),
    ("gemm.1x1s2.grid4.sub.bn.relux", 2, 3, 24, 16, 64, 1, 2, 0, 0, 0, 2, 24, 1, 2),
]


@pytest.mark.parametrize("case", DGRAD_EPILOGUE, ids=[c[0] for c in DGRAD_EPILOGUE])
def test_conv_data_gradient_epilogue(case):
    """One data-gradient launch with every epilogue operand, as cb_step uses
    it: accumulate, residual add (same shape or the option-A subsample),
    ReLU mask, and the fused batch-norm backward partial sums, against the
    oracle's data gradient with the epilogue applied by plain numpy."""
    name, k, b, Ci, H, Co, R, st, pad, acc, use_mask, add_mode, add_C, bn, use_y = case
    Ho = (H + 2 * pad - R) // st + 1
    rng = _rng("dgrad" + name)
    N = k * b
    nw = Co * Ci * R * R
    pstride = nw + 5
    params = np.zeros(k * pstride, dtype=np.float32)
    for j in range(k):
        params[j * pstride:j * pstride + nw] = rng.standard_normal(nw) * np.sqrt(2.0 / (Ci * R * R))
    dy = rng.standard_normal((N, Co, Ho, Ho), dtype=np.float32)
    dx0 = rng.standard_normal((N, Ci, H, H), dtype=np.float32)
    mask = rng.standard_normal((N, Ci, H, H), dtype=np.float32) if use_mask else None
    add = None
    if add_mode == 1:
        add = rng.standard_normal((N, Ci, H, H), dtype=np.float32)
    elif add_mode == 2:
        add = rng.standard_normal((N, add_C, Ho, Ho), dtype=np.float32)
    bn_x = rng.standard_normal((N, Ci, H, H), dtype=np.float32) if bn else None
    bn_y = rng.standard_normal((N, Ci, H, H), dtype=np.float32) if (bn and use_y == 1) else None
    mean = (rng.standard_normal((k, Ci)) * 0.1).astype(np.float32) if bn else None
    istd = (rng.uniform(0.5, 2.0, (k, Ci))).astype(np.float32) if bn else None
    # use_y == 2: gamma and beta are given too, and bn_y is the sign of the
    # norm's output recomputed from bn_x, so reading it and recomputing it
    # must give the same mask
    gb = np.zeros(k * pstride, dtype=np.float32)
    for j in range(k):
        gb[j * pstride:j * pstride + Ci] = 1 + 0.3 * rng.standard_normal(Ci)
        gb[j * pstride + Ci:j * pstride + 2 * Ci] = 0.5 * rng.standard_normal(Ci)
    if bn and use_y in (2, 3):
        sign = np.concatenate([np.where(
            _bn_relu_from_x(bn_x[j * b:(j + 1) * b], mean[j], istd[j],
                            gb[j * pstride:j * pstride + Ci],
                            gb[j * pstride + Ci:j * pstride + 2 * Ci]), 1.0, -1.0)
            for j in range(k)]).astype(np.float32)
        if use_y == 2:
            bn_y = sign
        else:
            mask = sign
    L = cb.lib()
    parts = L.cb_test_conv_dgrad_parts(k, b, Ci, H, H, Co, R, st, pad)
    assert parts > 0
    d = {n_: (_dev(v) if v is not None else None) for n_, v in
         dict(dy=dy, p=params, dx=dx0, mask=mask, add=add, x=bn_x, y=bn_y, mean=mean,
              istd=istd, g=gb if (bn and use_y in (2, 3)) else None).items()}
    part = torch.zeros(k * Ci * parts * 2, dtype=torch.float64, device="cuda") if bn else None
    ptr = lambda t: t.data_ptr() if t is not None else None
    rc = L.cb_test_conv_dgrad(k, b, Ci, H, H, Co, R, st, pad, ptr(d["dy"]), ptr(d["p"]), pstride,
                              ptr(d["dx"]), acc, ptr(d["mask"]), ptr(d["add"]), add_mode, add_C,
                              ptr(d["x"]), ptr(d["y"]), ptr(d["mean"]), ptr(d["istd"]),
                              ptr(d["g"]), ptr(part), torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    got = d["dx"].cpu().numpy()
    sums = part.cpu().numpy().reshape(k, Ci, parts, 2).sum(axis=2) if bn else None
    for j in range(k):
        sl = slice(j * b, (j + 1) * b)
        w = params[j * pstride:j * pstride + nw].reshape(Co, Ci, R, R)
        _, ref, _, _ = oracle.conv2d(np.zeros((b, Ci, H, H), np.float32), w, None, st, pad,
                                     dy=dy[sl])
        if acc:
            ref = ref + dx0[sl]
        if add_mode == 1:
            ref = ref + add[sl]
        elif add_mode == 2:
            ref[:, :, ::st, ::st] += add[sl][:, :Ci]
        if use_mask:
            ref = np.where(mask[sl] > 0, ref, 0.0)
        assert max_rel(got[sl], ref) <= TOL_STEP1, (name, j, "dx")
        if bn:
            dd = ref if bn_y is None else np.where(bn_y[sl] > 0, ref, 0.0)
            xh = (bn_x[sl].astype(np.float64) - mean[j][None, :, None, None]) * \
                istd[j][None, :, None, None]
            s1 = dd.sum(axis=(0, 2, 3))
            s2 = (dd * xh).sum(axis=(0, 2, 3))
            assert max_rel(sums[j, :, 0], s1) <= TOL_STEP1, (name, j, "sum d")
            assert max_rel(sums[j, :, 1], s2) <= TOL_STEP1, (name, j, "sum d*xh")

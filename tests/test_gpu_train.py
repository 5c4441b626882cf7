"""GPU parity of the steps either side of the convolutions (Sec. 4.1, Fig. 2)
against the CPU oracle: batch normalisation + residual + ReLU forward with
Q_a, its backward with Q_e, and FP32 SGD with Q_w.  INT16 tensors, exponents,
flags and the exact channel sums bit-exact; every FP32 output (z, mean,
inv_std, dy, dres, dgamma, dbeta, w, v) within the 1e-6 relative bound and
expected at 0 ulp, since both sides take the same IEEE operations in the
same order."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, assert_fp32_close, note, to_dev, ulp_diff
from paper_1802_00930_amd import dfp

pytestmark = pytest.mark.gpu


def scale_with_exp(e):
    s = dfp.new_scale(DEV)
    s[1] = int(e)
    return s


def bn_inputs(seed, N, C, HW, ey=-12, with_res=False, bits=15):
    rng = np.random.default_rng(seed)
    lim = (1 << (bits - 2)) if bits == 15 else 32767
    y = rng.integers(-lim, lim + 1, (N, C, HW)).astype(np.int16)
    y[:, 0] = 1234 if C > 1 else y[:, 0]  # a constant channel (zero variance) when there are several
    gamma = rng.uniform(-2, 2, C).astype(np.float32)
    if C > 2:
        gamma[1] = 0.0
    beta = rng.uniform(-1, 1, C).astype(np.float32)
    res = rng.standard_normal((N, C, HW)).astype(np.float32) if with_res else None
    return y, ey, gamma, beta, res


def gpu_bn_fwd(y, ey, gamma, beta, res, eps, bits, rounding, seed):
    N, C, HW = y.shape
    d = dfp.make_bn_desc(N, C, HW, bits=bits, rounding=rounding, eps=eps, seed=seed)
    yt = to_dev(y)
    z = torch.empty(y.shape, dtype=torch.float32, device=DEV)
    zq = torch.empty(y.shape, dtype=torch.int16, device=DEV)
    sz = dfp.new_scale(DEV)
    mean = torch.empty(C, dtype=torch.float32, device=DEV)
    inv = torch.empty(C, dtype=torch.float32, device=DEV)
    sums = torch.empty((C, 2), dtype=torch.int64, device=DEV)
    ws = dfp.alloc_bn_workspace(d, DEV)
    dfp.dfp_bn_relu_fwd(d, yt, scale_with_exp(ey), to_dev(gamma), to_dev(beta), zq, sz, mean, inv,
                        res=to_dev(res) if res is not None else None, z=z, sums=sums, workspace=ws)
    torch.cuda.synchronize()
    return dict(z=z.cpu().numpy(), zq=zq.cpu().numpy(), sc=dfp.read_scale(sz), mean=mean.cpu().numpy(),
                inv_std=inv.cpu().numpy(), sums=sums.cpu().numpy())


def check_fwd(g, o, what):
    assert g["sc"]["exp"] == o["ez"] and g["sc"]["flags"] == o["flags"], (what, g["sc"], o["ez"], o["flags"])
    assert np.array_equal(g["sums"], o["sums"]), what
    assert np.array_equal(g["mean"].view(np.uint32), o["mean"].view(np.uint32)), what
    assert np.array_equal(g["inv_std"].view(np.uint32), o["inv_std"].view(np.uint32)), what
    assert_fp32_close(g["z"], o["z"], what + " z")
    assert ulp_diff(g["z"], o["z"]) == 0, what
    bad = np.nonzero(g["zq"].reshape(-1) != o["zq"].reshape(-1))[0]
    assert bad.size == 0, "%s zq mismatch at %s" % (what, bad[:5])


# (N, C, HW): hw multiples of 8 take the 16-byte statistics path; odd hw puts a
# Philox group of four across channels; the last two are ResNet-50 BN shapes
SHAPES = [(1, 1, 1), (2, 3, 1), (2, 6, 35), (3, 5, 49), (4, 8, 64), (2, 4, 6), (5, 7, 13), (32, 64, 3136),
          (64, 256, 196)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("with_res", [False, True])
def test_bn_forward(shape, with_res):
    N, C, HW = shape
    for bits, rounding in ((15, 0), (15, 1), (16, 2), (15, 3)):
        seed = 1000 + N * 7 + C + HW + rounding
        y, ey, gamma, beta, res = bn_inputs(seed, N, C, HW, with_res=with_res, bits=bits)
        note("bn fwd %s res=%d bits=%d rounding=%d" % (shape, with_res, bits, rounding))
        g = gpu_bn_fwd(y, ey, gamma, beta, res, 1e-5, bits, rounding, seed)
        o = oracle.bn_relu_fwd(y.reshape(N, C, HW, 1), ey, gamma, beta,
                               res.reshape(N, C, HW, 1) if res is not None else None, eps=1e-5, bits=bits,
                               rounding=rounding, seed=seed)
        check_fwd(g, o, "fwd %s res=%d bits=%d mode=%d" % (shape, with_res, bits, rounding))


@pytest.mark.parametrize("ey,eps", [(-128, 1e-5), (-128, 0.0), (20, 1e-3), (-30, 0.0)])
def test_bn_forward_exponent_extremes(ey, eps):
    # tiny and large values, eps = 0 (a constant channel then has inv_std = inf)
    y, _, gamma, beta, _ = bn_inputs(7, 3, 5, 40)
    y[:, 2] = 0
    note("bn fwd ey=%d eps=%g" % (ey, eps))
    g = gpu_bn_fwd(y, ey, gamma, beta, None, eps, 15, 1, 5)
    o = oracle.bn_relu_fwd(y.reshape(3, 5, 40, 1), ey, gamma, beta, None, eps=eps, bits=15, rounding=1, seed=5)
    check_fwd(g, o, "ey=%d eps=%g" % (ey, eps))


def test_bn_forward_all_negative_is_zero_tensor():
    y, ey, gamma, beta, _ = bn_inputs(8, 2, 4, 16)
    beta[:] = -100.0
    g = gpu_bn_fwd(y, ey, gamma, beta, None, 1e-5, 15, 0, 0)
    o = oracle.bn_relu_fwd(y.reshape(2, 4, 16, 1), ey, gamma, beta, None)
    assert o["flags"] == oracle.FLAG_ZERO_TENSOR
    check_fwd(g, o, "all negative")


def gpu_bn_bwd(dz, edz, y, ey, gamma, beta, mean, inv, res, bits, rounding, seed, eps=1e-5):
    N, C, HW = y.shape
    d = dfp.make_bn_desc(N, C, HW, bits=bits, rounding=rounding, eps=eps, seed=seed)
    dy = torch.empty(y.shape, dtype=torch.float32, device=DEV)
    dyq = torch.empty(y.shape, dtype=torch.int16, device=DEV)
    sdy = dfp.new_scale(DEV)
    dg = torch.empty(C, dtype=torch.float32, device=DEV)
    db = torch.empty(C, dtype=torch.float32, device=DEV)
    dres = torch.empty(y.shape, dtype=torch.float32, device=DEV) if res is not None else None
    sums = torch.empty((C, 2), dtype=torch.int64, device=DEV)
    ws = dfp.alloc_bn_workspace(d, DEV)
    dfp.dfp_bn_relu_bwd(d, to_dev(dz), scale_with_exp(edz), to_dev(y), scale_with_exp(ey), to_dev(gamma),
                        to_dev(beta), to_dev(mean), to_dev(inv), dyq, sdy, dg, db,
                        res=to_dev(res) if res is not None else None, dy=dy, dres=dres, sums=sums, workspace=ws)
    torch.cuda.synchronize()
    return dict(dy=dy.cpu().numpy(), dyq=dyq.cpu().numpy(), sc=dfp.read_scale(sdy), dgamma=dg.cpu().numpy(),
                dbeta=db.cpu().numpy(), dres=dres.cpu().numpy() if dres is not None else None,
                sums=sums.cpu().numpy())


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("with_res", [False, True])
def test_bn_backward(shape, with_res):
    N, C, HW = shape
    for bits, rounding in ((15, 1), (15, 0), (16, 2)):
        seed = 2000 + N * 7 + C + HW + rounding
        y, ey, gamma, beta, res = bn_inputs(seed, N, C, HW, with_res=with_res, bits=bits)
        r4 = res.reshape(N, C, HW, 1) if res is not None else None
        fw = oracle.bn_relu_fwd(y.reshape(N, C, HW, 1), ey, gamma, beta, r4)
        rng = np.random.default_rng(seed + 1)
        dz = rng.integers(-16384, 16385, y.shape).astype(np.int16)
        edz = -24
        note("bn bwd %s res=%d bits=%d rounding=%d" % (shape, with_res, bits, rounding))
        g = gpu_bn_bwd(dz, edz, y, ey, gamma, beta, fw["mean"], fw["inv_std"], res, bits, rounding, seed)
        o = oracle.bn_relu_bwd(dz.reshape(N, C, HW, 1), edz, y.reshape(N, C, HW, 1), ey, gamma, beta, fw["mean"],
                               fw["inv_std"], r4, bits=bits, rounding=rounding, seed=seed)
        what = "bwd %s res=%d bits=%d mode=%d" % (shape, with_res, bits, rounding)
        assert g["sc"]["exp"] == o["edy"] and g["sc"]["flags"] == o["flags"], (what, g["sc"], o["edy"])
        assert np.array_equal(g["sums"], o["sums"]), what
        assert np.array_equal(g["dgamma"].view(np.uint32), o["dgamma"].view(np.uint32)), what
        assert np.array_equal(g["dbeta"].view(np.uint32), o["dbeta"].view(np.uint32)), what
        assert_fp32_close(g["dy"], o["dy"], what + " dy")
        assert ulp_diff(g["dy"], o["dy"]) == 0, what
        if with_res:
            assert np.array_equal(g["dres"].reshape(-1).view(np.uint32), o["dres"].reshape(-1).view(np.uint32))
        bad = np.nonzero(g["dyq"].reshape(-1) != o["dyq"].reshape(-1))[0]
        assert bad.size == 0, "%s dyq mismatch at %s" % (what, bad[:5])


def test_bn_backward_zero_gradient():
    y, ey, gamma, beta, _ = bn_inputs(9, 2, 4, 16)
    fw = oracle.bn_relu_fwd(y.reshape(2, 4, 16, 1), ey, gamma, beta)
    g = gpu_bn_bwd(np.zeros_like(y), 0, y, ey, gamma, beta, fw["mean"], fw["inv_std"], None, 15, 0, 0)
    assert g["sc"]["flags"] == oracle.FLAG_ZERO_TENSOR and g["sc"]["exp"] == 0
    assert not g["dyq"].any() and not g["dy"].any() and not g["dgamma"].any() and not g["dbeta"].any()


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1000, 36864, 589824, 2359296 + 3])
def test_sgd_two_steps(n):
    rng = np.random.default_rng(n)
    w0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    v0 = np.zeros(n, np.float32)
    wt, vt = to_dev(w0), to_dev(v0)
    w, v = w0, v0
    for step, (rounding, bits) in enumerate(((1, 15), (0, 16))):
        dw = (rng.standard_normal(n) * 1e-3).astype(np.float32)
        wq = torch.empty(n, dtype=torch.int16, device=DEV)
        sw = dfp.new_scale(DEV)
        note("sgd n=%d step=%d" % (n, step))
        dfp.dfp_sgd_quantize(0.1, 0.9, 1e-4, bits, rounding, 77 + step, wt, vt, to_dev(dw), wq, sw)
        torch.cuda.synchronize()
        o = oracle.sgd_quantize(w, v, dw, 0.1, 0.9, 1e-4, bits=bits, rounding=rounding, seed=77 + step)
        w, v = o["w"], o["v"]
        assert np.array_equal(wt.cpu().numpy().view(np.uint32), w.view(np.uint32)), step
        assert np.array_equal(vt.cpu().numpy().view(np.uint32), v.view(np.uint32)), step
        sc = dfp.read_scale(sw)
        assert sc["exp"] == o["ew"] and sc["flags"] == o["flags"], (sc, o["ew"], o["flags"])
        assert np.array_equal(wq.cpu().numpy(), o["wq"]), step

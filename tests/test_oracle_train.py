"""Pins of the oracle's training-step pieces around the convolutions (Sec.
4.1, Fig. 2) against references outside it: PyTorch's float64 batch
normalisation (training mode) with ReLU and a residual add, its autograd
backward, torch.optim.SGD with momentum and weight decay, numpy int64 channel
sums, and the property that the forward output's max is reached at a
channel's smallest or largest input integer."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def layer(seed, N=4, C=6, H=5, W=7, ey=-12):
    rng = np.random.default_rng(seed)
    y = rng.integers(-16384, 16385, (N, C, H, W)).astype(np.int16)
    y[:, 0] = 1234  # a constant channel: zero variance
    gamma = rng.uniform(-2, 2, C).astype(np.float32)
    gamma[1] = 0.0
    beta = rng.uniform(-1, 1, C).astype(np.float32)
    return y, ey, gamma, beta


def torch_bn_relu(y, ey, gamma, beta, res, eps):
    yt = torch.tensor(np.ldexp(y.astype(np.float64), ey), requires_grad=True)
    rt = torch.tensor(res.astype(np.float64), requires_grad=True) if res is not None else None
    pre = F.batch_norm(yt, None, None, torch.tensor(gamma, dtype=torch.float64),
                       torch.tensor(beta, dtype=torch.float64), training=True, eps=eps)
    if rt is not None:
        pre = pre + rt
    return yt, rt, pre, torch.relu(pre)


@pytest.mark.parametrize("with_res", [False, True])
def test_forward_matches_torch_float64(with_res):
    y, ey, gamma, beta = layer(1)
    res = np.random.default_rng(2).standard_normal(y.shape).astype(np.float32) if with_res else None
    o = oracle.bn_relu_fwd(y, ey, gamma, beta, res, eps=1e-5)
    _, _, pre, z = torch_bn_relu(y, ey, gamma, beta, res, 1e-5)
    z = z.detach().numpy()
    assert np.allclose(o["z"], z, rtol=1e-5, atol=1e-5)
    # exact integer sums and the float64 statistics
    yi = y.astype(np.int64)
    assert np.array_equal(o["sums"][:, 0], yi.sum(axis=(0, 2, 3)))
    assert np.array_equal(o["sums"][:, 1], (yi * yi).sum(axis=(0, 2, 3)))
    yv = np.ldexp(y.astype(np.float64), ey)
    assert np.array_equal(o["mean"], yv.mean(axis=(0, 2, 3)).astype(np.float32))
    inv = 1.0 / np.sqrt(yv.var(axis=(0, 2, 3)) + 1e-5)
    assert np.allclose(o["inv_std"], inv, rtol=1e-6)
    # Q_a of z is the single-exponent quantiser on z
    rq, re, rfl = oracle.quantize(o["z"], 15, oracle.ROUND_NEAREST, 0, oracle.ROLE_X)
    assert np.array_equal(o["zq"], rq) and o["ez"] == re and o["flags"] == rfl


def test_forward_max_sits_at_a_channel_extreme():
    # per channel the output is a monotone function of the input integer, so
    # its max over the tensor is reached at some channel's smallest or largest
    # integer (this is what lets a kernel quantise the output in one pass)
    for seed in range(5):
        y, ey, gamma, beta = layer(10 + seed)
        o = oracle.bn_relu_fwd(y, ey, gamma, beta)
        per_channel = []
        for c in range(y.shape[1]):
            zc, yc = o["z"][:, c], y[:, c]
            ext = max(zc[yc == yc.min()].max(), zc[yc == yc.max()].max())
            assert zc.max() == ext
            per_channel.append(ext)
        assert o["z"].max() == max(per_channel)


@pytest.mark.parametrize("with_res", [False, True])
def test_backward_matches_torch_autograd(with_res):
    y, ey, gamma, beta = layer(3)
    rng = np.random.default_rng(4)
    res = rng.standard_normal(y.shape).astype(np.float32) if with_res else None
    fw = oracle.bn_relu_fwd(y, ey, gamma, beta, res, eps=1e-5)
    dz = rng.integers(-16384, 16385, y.shape).astype(np.int16)
    edz = -20
    o = oracle.bn_relu_bwd(dz, edz, y, ey, gamma, beta, fw["mean"], fw["inv_std"], res)
    yt, rt, pre, z = torch_bn_relu(y, ey, gamma, beta, res, 1e-5)
    dzt = torch.tensor(np.ldexp(dz.astype(np.float64), edz))
    # the oracle's ReLU mask comes from its FP32 pre-activation; use it in the
    # reference too (elements where the two pre-activations differ in sign sit at 0)
    mask = fw["z"] > 0
    pre64 = pre.detach().numpy()
    assert np.all((pre64 > 0) == mask) or np.abs(pre64[(pre64 > 0) != mask]).max() < 1e-5
    g64 = torch.autograd.grad(pre, [yt] + ([rt] if rt is not None else []), grad_outputs=dzt * torch.tensor(mask))
    ref_dy = g64[0].numpy()
    scale = np.abs(ref_dy).max()
    assert np.abs(o["dy"] - ref_dy).max() <= 1e-5 * scale
    yv = torch.tensor(np.ldexp(y.astype(np.float64), ey))
    xhat = (yv - yv.mean(dim=(0, 2, 3), keepdim=True)) / torch.sqrt(yv.var(dim=(0, 2, 3), unbiased=False,
                                                                            keepdim=True) + 1e-5)
    dzm = dzt * torch.tensor(mask)
    assert np.allclose(o["dbeta"], dzm.sum(dim=(0, 2, 3)).numpy(), rtol=1e-6, atol=1e-12)
    assert np.allclose(o["dgamma"], (dzm * xhat).sum(dim=(0, 2, 3)).numpy(), rtol=1e-5, atol=1e-9)
    # exact masked integer sums
    gi = np.where(mask, dz.astype(np.int64), 0)
    assert np.array_equal(o["sums"][:, 0], gi.sum(axis=(0, 2, 3)))
    assert np.array_equal(o["sums"][:, 1], (gi * y.astype(np.int64)).sum(axis=(0, 2, 3)))
    if with_res:
        assert np.array_equal(o["dres"], np.where(mask, np.ldexp(dz.astype(np.float32), edz), 0).astype(np.float32))
    rq, re, rfl = oracle.quantize(o["dy"], 15, oracle.ROUND_NEAREST, 0, oracle.ROLE_DY)
    assert np.array_equal(o["dyq"], rq) and o["edy"] == re


def test_zero_gradient_gives_zero_outputs():
    y, ey, gamma, beta = layer(5)
    fw = oracle.bn_relu_fwd(y, ey, gamma, beta)
    o = oracle.bn_relu_bwd(np.zeros_like(y), 0, y, ey, gamma, beta, fw["mean"], fw["inv_std"])
    assert not o["dy"].any() and not o["dyq"].any() and o["flags"] == oracle.FLAG_ZERO_TENSOR
    assert not o["dgamma"].any() and not o["dbeta"].any()


def test_sgd_matches_torch_optim():
    rng = np.random.default_rng(6)
    w0 = rng.standard_normal(1000).astype(np.float32)
    wt = torch.tensor(w0.astype(np.float64), requires_grad=True)
    opt = torch.optim.SGD([wt], lr=0.1, momentum=0.9, weight_decay=1e-4)
    w, v = w0.copy(), np.zeros_like(w0)
    for step in range(3):
        dw = rng.standard_normal(1000).astype(np.float32)
        o = oracle.sgd_quantize(w, v, dw, 0.1, 0.9, 1e-4)
        w, v = o["w"], o["v"]
        wt.grad = torch.tensor(dw.astype(np.float64))
        opt.step()
        assert np.allclose(w, wt.detach().numpy(), rtol=1e-5, atol=1e-6), step
        rq, re, _ = oracle.quantize(w, 15, oracle.ROUND_NEAREST, 0, oracle.ROLE_W)
        assert np.array_equal(o["wq"], rq) and o["ew"] == re

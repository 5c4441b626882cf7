"""dfp_conv_bwd_weights_noalloc: the backward-weights convolution with its
scratch in the library's static device array instead of a caller workspace.

Through the C ABI, every call is compared bit for bit with
dfp_conv_bwd_weights on the same quantised operands (with a workspace the
caller allocates), on consecutive calls whose layers shrink, so that each
call runs on scratch still holding the previous call's contents.  The last,
smallest layer is also checked against the CPU oracle.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, GpuLayer, note, oracle_geom
from paper_1802_00930_amd import dfp
from paper_1802_00930_amd.workloads import WORKLOADS, layer_inputs

pytestmark = pytest.mark.gpu

# (label, n, c, h, w, k, r, s, stride, pad, L, G, rounding, seed); each needs at
# most 64 MiB of scratch, in decreasing size
SEQUENCE = (
    ("conv2_x 3x3 N=32 (benchmark layer)", 32, 64, 56, 56, 64, 3, 3, 1, 1, 64, 16, "stochastic", 1),
    ("3x3 N=8, 40 channels, 30x30", 8, 40, 30, 30, 48, 3, 3, 1, 1, 64, 16, "nearest", 7),
    ("strided 1x1 N=4 256->128 14x14 s2", 4, 256, 14, 14, 128, 1, 1, 2, 0, 64, 16, "biased", 3),
    ("unit 1x1 N=2 64->96 28x28", 2, 64, 28, 28, 96, 1, 1, 1, 0, 64, 16, "nearest", 5),
    ("3x3 N=2 16->32 14x14, L=16", 2, 16, 14, 14, 32, 3, 3, 1, 1, 16, 0, "nearest", 0),
)


def _inputs(label, n, c, h, w, k, r, s, stride, pad, rounding, seed, gl):
    rng = np.random.default_rng(zlib.crc32(label.encode()))
    x = np.maximum(rng.standard_normal(gl.shape_x, dtype=np.float32), 0)
    wt = rng.standard_normal(gl.shape_w, dtype=np.float32) * np.float32(np.sqrt(2.0 / (c * r * s)))
    dy = rng.standard_normal(gl.shape_y, dtype=np.float32) * np.float32(1e-3)
    return x, wt, dy


def test_noalloc_matches_workspace_call_on_shrinking_layers():
    for i, (label, n, c, h, w, k, r, s, stride, pad, L, G, rounding, seed) in enumerate(SEQUENCE):
        gl = GpuLayer(n, c, h, w, k, r, s, stride, pad, L=L, rounding=rounding, seed=seed, G=G)
        need = dfp.workspace_bytes(gl.d, dfp.BWD_WT)
        assert 0 < need <= dfp.NOALLOC_SCRATCH_BYTES, (label, need)
        note("noalloc %d: %s (scratch %d bytes)" % (i, label, need))
        x, wt, dy = _inputs(label, n, c, h, w, k, r, s, stride, pad, rounding, seed, gl)
        qx, sx = gl.quantize(x, dfp.ROLE_X)
        qdy, sdy = gl.quantize(dy, dfp.ROLE_DY)
        ref, _, _ = gl.conv(dfp.BWD_WT, qx, sx, qdy, sdy)
        got = torch.full(gl.shape_w, float("nan"), dtype=torch.float32, device=DEV)
        dfp.dfp_conv_bwd_weights_noalloc(gl.d, qx, sx, qdy, sdy, got)
        torch.cuda.synchronize()
        a, b = got.cpu().numpy(), ref.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "%s: %d elements differ" % (
            label, np.count_nonzero(a.view(np.uint32) != b.view(np.uint32)))
        if i == len(SEQUENCE) - 1:
            g = oracle_geom(gl)
            ox = qx.cpu().numpy()
            ody = qdy.cpu().numpy()
            e = dfp.read_scale(sx)["exp"] + dfp.read_scale(sdy)["exp"]
            o, _, _ = oracle.conv(g, oracle.BWD_WT, ox, ody, e, L, G if G > 0 else oracle.default_seg_chunks(L))
            assert np.array_equal(a.reshape(-1).view(np.uint32), o.reshape(-1).view(np.uint32))
        del ref, got


def test_noalloc_twice_on_the_benchmark_layer_then_smaller():
    """Two calls in a row on the benchmark workload's own inputs, then one on a
    batch of 4 of the same layer: each equals the workspace call."""
    wl = WORKLOADS["resnet50_conv2x_3x3"]
    for n in (32, 32, 4):
        layer, x, w, dy = layer_inputs(wl, 0, scale_n=n)
        gl = GpuLayer(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad, L=64,
                      rounding="stochastic", seed=wl.seed, G=16)
        note("noalloc benchmark layer N=%d" % n)
        qx, sx = gl.quantize(x, dfp.ROLE_X)
        qdy, sdy = gl.quantize(dy, dfp.ROLE_DY)
        ref, _, _ = gl.conv(dfp.BWD_WT, qx, sx, qdy, sdy)
        got = torch.empty(gl.shape_w, dtype=torch.float32, device=DEV)
        dfp.dfp_conv_bwd_weights_noalloc(gl.d, qx, sx, qdy, sdy, got)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int32), ref.view(torch.int32))


def test_noalloc_rejects_layer_beyond_scratch():
    wl = WORKLOADS["vgg16_conv1_2_conv3_3"]
    layer = wl.layers[0]
    d = dfp.make_desc(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad,
                      chunk_len=64, seg_chunks=16)
    assert dfp.workspace_bytes(d, dfp.BWD_WT) > dfp.NOALLOC_SCRATCH_BYTES
    t16 = torch.zeros(16, dtype=torch.int16, device=DEV)
    sc = dfp.new_scale(DEV)
    out = torch.zeros(16, dtype=torch.float32, device=DEV)
    with pytest.raises(dfp.DfpError) as ei:
        dfp.dfp_conv_bwd_weights_noalloc(d, t16, sc, t16, sc, out)
    assert ei.value.status == dfp.ERR_SCRATCH_LIMIT

"""GPU parity at the full sizes of the benchmark workloads, in the launch
configuration the benchmark times (default path, chunk lengths of the
workload, default backward-weights segments unless stated).

Every quantisation is compared in full (INT16 bit-exact, exponents and flags
equal).  Convolution outputs are compared in full where the oracle finishes
in seconds (the ResNet-50 conv2_x 3x3 layer at L = 64, the configuration of
the headline number) and otherwise at sampled output elements, each computed
one by one by the oracle, together with their INT32 chunk partials.  The
down-convert is checked in full against the oracle's quantiser applied to the
GPU's FP32 output, and the convolution epilogue's max |y| against the output
itself.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, GpuLayer, assert_fp32_close, note, oracle_geom, ulp_diff
from paper_1802_00930_amd import dfp
from paper_1802_00930_amd.workloads import WORKLOADS, layer_inputs

pytestmark = pytest.mark.gpu

DIRS = (dfp.FWD, dfp.BWD_DATA, dfp.BWD_WT)


def _quantize_both(gl, f, role, bits, rounding, seed):
    q, sc = gl.quantize(f, role)
    oq, oe, oflags = oracle.quantize(f, bits, oracle.ROUNDING[rounding], seed, role)
    torch.cuda.synchronize()
    got = q.cpu().numpy()
    bad = np.count_nonzero(got != oq)
    assert bad == 0, "quantise role %d: %d elements differ" % (role, bad)
    s = dfp.read_scale(sc)
    assert s["exp"] == oe and s["flags"] == oflags, (role, s, oe, oflags)
    return q, sc, oq, oe


def check_layer(layer, x, w, dy, L, rounding, seed, nsample=0, G=0, dirs=DIRS, partial_samples=64):
    """Quantise, run the three convolutions and both down-converts of one layer
    on the GPU; compare with the oracle.  nsample = 0: every output element."""
    gl = GpuLayer(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad, L=L,
                  rounding=rounding, seed=seed, G=G)
    g = oracle_geom(gl)
    Gd = G if G > 0 else oracle.default_seg_chunks(L)
    note("layer %s N=%d L=%d %s: quantise" % (layer.name, layer.n, L, rounding))
    qx, sx, ox, ex = _quantize_both(gl, x, dfp.ROLE_X, 15, rounding, seed)
    qw, sw, ow, ew = _quantize_both(gl, w, dfp.ROLE_W, 15, rounding, seed)
    qdy, sdy, ody, edy = _quantize_both(gl, dy, dfp.ROLE_DY, 15, rounding, seed)
    rng = np.random.default_rng(zlib.crc32(("%s/%d/%s" % (layer.name, L, rounding)).encode()))
    operands = {dfp.FWD: (qx, sx, qw, sw, ox, ow, ex + ew),
                dfp.BWD_DATA: (qdy, sdy, qw, sw, ody, ow, edy + ew),
                dfp.BWD_WT: (qx, sx, qdy, sdy, ox, ody, ex + edy)}
    for direction in dirs:
        a, sa, b, sb, oa, ob, e = operands[direction]
        note("layer %s dir %d: conv" % (layer.name, direction))
        out, so, _ = gl.conv(direction, a, sa, b, sb)
        torch.cuda.synchronize()
        got = out.cpu().numpy().reshape(-1)
        if nsample == 0:
            ref, _, _ = oracle.conv(g, direction, oa, ob, e, L, Gd)
            ref = ref.reshape(-1)
            idx = None
        else:
            # backward-weights outputs each reduce over N*P*Q products: bound the oracle's work
            ns = nsample if direction != dfp.BWD_WT else max(64, min(nsample, int(2e8 // (g.n * gl.p * gl.q))))
            idx = np.unique(np.concatenate([rng.integers(0, got.size, ns), [0, got.size - 1]]))
            ref, _, _ = oracle.conv_at(g, direction, oa, ob, e, L, idx, Gd)
            got = got[idx]
        assert_fp32_close(got, ref, "%s dir %d" % (layer.name, direction))
        assert ulp_diff(got, ref) == 0
        # INT32 chunk partials at a few outputs, from a second call that records them
        if partial_samples:
            pidx = rng.integers(0, out.numel(), partial_samples)
            J = dfp.num_chunks(gl.d, direction)
            if J * out.numel() * 4 <= (4 << 30):
                _, _, parts = gl.conv(direction, a, sa, b, sb, want_scale=False, want_partials=True)
                gp = parts[:, torch.from_numpy(pidx).to(DEV)].cpu().numpy().T
                del parts
                _, rp, _ = oracle.conv_at(g, direction, oa, ob, e, L, pidx, Gd, want_partials=True)
                assert np.array_equal(gp, rp), "%s dir %d partials differ" % (layer.name, direction)
        if direction != dfp.BWD_WT:
            # epilogue max |y| and the down-convert of this output (role Y or DX)
            y = out.cpu().numpy()
            s = dfp.read_scale(so)
            assert s["amax_bits"] == int((y.view(np.uint32) & 0x7fffffff).max())
            role = dfp.ROLE_Y if direction == dfp.FWD else dfp.ROLE_DX
            qo, sq = gl.downconvert(out, role, so)
            oq, oe, oflags = oracle.quantize(y, 15, oracle.ROUNDING[rounding], seed, role)
            torch.cuda.synchronize()
            assert np.count_nonzero(qo.cpu().numpy() != oq) == 0, "%s down-convert differs" % layer.name
            assert dfp.read_scale(sq)["exp"] == oe
        del out


def test_resnet50_conv2x_3x3_full_l64():
    """N=32, 64->64 at 56x56, stochastic seed 1, L = 64: every output of all
    three convolutions (the benchmark's workload and launch configuration)."""
    wl = WORKLOADS["resnet50_conv2x_3x3"]
    layer, x, w, dy = layer_inputs(wl, 0)
    check_layer(layer, x, w, dy, 64, "stochastic", wl.seed, nsample=0, G=16)


@pytest.mark.parametrize("L", [8, 16, 32])
def test_resnet50_conv2x_3x3_chunk_sweep(L):
    wl = WORKLOADS["resnet50_conv2x_3x3"]
    layer, x, w, dy = layer_inputs(wl, 0)
    check_layer(layer, x, w, dy, L, "stochastic", wl.seed, nsample=20000, G=max(1, 16 * 64 // L))


@pytest.mark.parametrize("rounding", ["nearest", "biased"])
def test_resnet50_conv4x_1x1_pair(rounding):
    wl = WORKLOADS["resnet50_conv4x_1x1"]
    for i in range(len(wl.layers)):
        layer, x, w, dy = layer_inputs(wl, i)
        check_layer(layer, x, w, dy, 64, rounding, wl.seed, nsample=20000)


def test_vgg16_conv1_2_conv3_3():
    wl = WORKLOADS["vgg16_conv1_2_conv3_3"]
    for i in range(len(wl.layers)):
        layer, x, w, dy = layer_inputs(wl, i)
        check_layer(layer, x, w, dy, 64, "stochastic", wl.seed, nsample=4000, partial_samples=16)


def test_resnet50_all_53_layers():
    """Every ResNet-50 convolution (7x7 stem, strided 1x1 and projection
    shortcuts, 3x3 bottlenecks) at N=64, nearest, L = 64, sampled outputs."""
    wl = WORKLOADS["resnet50_all_convs"]
    assert len(wl.layers) == 53
    for i in range(len(wl.layers)):
        layer, x, w, dy = layer_inputs(wl, i)
        check_layer(layer, x, w, dy, 64, "nearest", wl.seed, nsample=1500, partial_samples=8)
        torch.cuda.empty_cache()


def test_resnet50_conv2x_3x3_dfp32_full():
    """The same layer through the single-chunk DFP-32 outputs (forward and
    backward-data at L = C*R*S = K*R*S = 576) and the integer down-convert
    with the epilogue's max, every element against the oracle."""
    wl = WORKLOADS["resnet50_conv2x_3x3"]
    layer, x, w, dy = layer_inputs(wl, 0)
    L = layer.c * layer.r * layer.s
    gl = GpuLayer(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad, L=L,
                  rounding="stochastic", seed=wl.seed)
    g = oracle_geom(gl)
    rnd = oracle.ROUNDING["stochastic"]
    qx, sx, ox, ex = _quantize_both(gl, x, dfp.ROLE_X, 15, "stochastic", wl.seed)
    qw, sw, ow, ew = _quantize_both(gl, w, dfp.ROLE_W, 15, "stochastic", wl.seed)
    qdy, sdy, ody, edy = _quantize_both(gl, dy, dfp.ROLE_DY, 15, "stochastic", wl.seed)
    for direction, a, sa, oa, ea, role, shape in ((dfp.FWD, qx, sx, ox, ex, dfp.ROLE_Y, gl.shape_y),
                                                  (dfp.BWD_DATA, qdy, sdy, ody, edy, dfp.ROLE_DX, gl.shape_x)):
        note("dfp32 layer %s dir %d" % (layer.name, direction))
        out = torch.empty(shape, dtype=torch.int32, device=DEV)
        so = dfp.new_scale(DEV)
        ws = dfp.alloc_workspace(gl.d, direction, DEV)
        f = dfp.dfp_conv_fwd_i32 if direction == dfp.FWD else dfp.dfp_conv_bwd_data_i32
        f(gl.d, a, sa, qw, sw, out, so, ws)
        q = torch.empty(shape, dtype=torch.int16, device=DEV)
        sq = dfp.new_scale(DEV)
        dfp.dfp_downconvert_i32(gl.d, role, out, so, q, sq, amax_ready=True)
        _, rparts, _ = oracle.conv(g, direction, oa, ow, ea + ew, L, 1, want_partials=True)
        rq, re, rf = oracle.downconvert_i32(rparts[0], ea + ew, 15, rnd, wl.seed, role)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().reshape(-1), rparts[0])
        assert np.array_equal(q.cpu().numpy().reshape(-1), rq)
        s = dfp.read_scale(sq)
        assert (s["exp"], s["flags"]) == (re, rf)
        del out, q, ws

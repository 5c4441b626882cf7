"""GPU parity of the three DFP convolutions and the down-convert against the
CPU oracle on identical seeded inputs: INT32 chunk partials and INT16 tensors
bit-exact, exponents equal, FP32 outputs within 1e-6 relative (expected 0 ulp).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, GpuLayer, assert_fp32_close, note, oracle_geom, to_dev, ulp_diff
from paper_1802_00930_amd import dfp

pytestmark = pytest.mark.gpu

SHAPES = [
    # n, c, h, w, k, r, s, stride, pad
    (2, 16, 14, 14, 32, 3, 3, 1, 1),
    (2, 3, 9, 8, 4, 3, 3, 1, 1),
    (1, 5, 7, 7, 3, 1, 1, 1, 0),
    (2, 4, 10, 9, 5, 3, 3, 2, 1),
    (1, 3, 23, 23, 8, 7, 7, 2, 3),
    (2, 8, 6, 6, 6, 1, 1, 2, 0),
    (1, 2, 5, 6, 3, 3, 2, 1, 0),
    (1, 6, 4, 4, 2, 3, 3, 3, 2),
    (3, 64, 9, 11, 40, 3, 3, 1, 1),
    (2, 96, 7, 7, 130, 1, 1, 1, 0),
    (1, 70, 12, 12, 33, 3, 3, 2, 1),
]


def run_all(shape, L, path=dfp.PATH_AUTO, rounding="nearest", seed=0, G=0, scale=1.0, partials=True, bits=15,
            pad_w=None):
    n, c, h, w, k, r, s, st, pd = shape
    gl = GpuLayer(n, c, h, w, k, r, s, st, pd, L=L, bits=bits, rounding=rounding, seed=seed, path=path, G=G,
                  pad_w=pad_w)
    rng = np.random.default_rng(abs(hash((shape, L, seed))) % 2 ** 32)
    x = (rng.standard_normal(gl.shape_x) * scale).astype(np.float32)
    wt = (rng.standard_normal(gl.shape_w) * scale).astype(np.float32)
    dy = (rng.standard_normal(gl.shape_y) * scale).astype(np.float32)
    rnd = dfp.ROUNDING[rounding]
    qx, sx = gl.quantize(x, dfp.ROLE_X)
    qw, sw = gl.quantize(wt, dfp.ROLE_W)
    qdy, sdy = gl.quantize(dy, dfp.ROLE_DY)
    ox, ex, _ = oracle.quantize(x, bits, rnd, seed, oracle.ROLE_X)
    ow, ew, _ = oracle.quantize(wt, bits, rnd, seed, oracle.ROLE_W)
    ody, edy, _ = oracle.quantize(dy, bits, rnd, seed, oracle.ROLE_DY)
    torch.cuda.synchronize()
    assert np.array_equal(qx.cpu().numpy(), ox) and np.array_equal(qw.cpu().numpy(), ow)
    assert np.array_equal(qdy.cpu().numpy(), ody)
    g = oracle_geom(gl)
    Gd = G if G > 0 else oracle.default_seg_chunks(L)
    res = {}
    for direction, a, sa, b, sb, oa, ob, e in (
            (dfp.FWD, qx, sx, qw, sw, ox, ow, ex + ew),
            (dfp.BWD_DATA, qdy, sdy, qw, sw, ody, ow, edy + ew),
            (dfp.BWD_WT, qx, sx, qdy, sdy, ox, ody, ex + edy)):
        note("conv shape=%s L=%d dir=%d path=%d" % (shape, L, direction, path))
        out, so, parts = gl.conv(direction, a, sa, b, sb, want_partials=partials)
        ref, rparts, ov = oracle.conv(g, direction, oa, ob, e, L, Gd, want_partials=partials)
        torch.cuda.synchronize()
        if partials:
            gp = parts.cpu().numpy()
            bad = np.argwhere(gp != rparts)
            assert bad.size == 0, "partials differ dir=%d at %s" % (direction, bad[:5])
        got = out.cpu().numpy()
        assert_fp32_close(got, ref, "dir %d" % direction)
        assert ulp_diff(got, ref) == 0
        res[direction] = (gl, out, so, ref)
    return res


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("L", [1, 5, 8, 16, 64, 10 ** 7])
def test_small_shapes(shape, L):
    run_all(shape, L)


@pytest.mark.parametrize("path", [dfp.PATH_MFMA, dfp.PATH_VALU])
@pytest.mark.parametrize("L", [8, 16, 32, 64, 96, 128])
def test_paths_agree(path, L):
    for shape in ((2, 64, 10, 10, 64, 3, 3, 1, 1), (2, 128, 7, 7, 96, 1, 1, 1, 0), (1, 32, 9, 9, 64, 3, 3, 2, 1)):
        run_all(shape, L, path=path)


# Unit-stride layers whose output rows are a multiple of 8 wide and whose
# reduction length is a multiple of 32: the backward-weights band kernel
# (runs of 8 indices per output row) takes these, the other shapes above do not.
BAND_SHAPES = [
    (2, 16, 8, 8, 32, 3, 3, 1, 1),
    (1, 24, 16, 16, 40, 3, 3, 1, 1),
    (2, 8, 12, 24, 16, 1, 1, 1, 0),
    (4, 32, 7, 8, 20, 3, 3, 1, 1),
    (2, 64, 24, 16, 64, 3, 3, 1, 1),
    (2, 16, 10, 8, 80, 3, 3, 1, 1),  # dy digits: two 64-channel tiles, 160 indices (a partial 128-index tile)
]


@pytest.mark.parametrize("shape", BAND_SHAPES)
@pytest.mark.parametrize("L,G", [(32, 0), (64, 0), (64, 3), (128, 1), (64, 5)])
def test_bwd_wt_band_shapes(shape, L, G):
    run_all(shape, L, G=G)


# Strided 1x1 layers without padding (ResNet-50's downsampling projections):
# the weight gradient runs on the subsampled input with unit stride, so the
# MFMA path takes layers whose strided input band would not fit in LDS (the
# first shape), at odd sizes and stride 3 too; bit-exact against the oracle's
# strided sum.
@pytest.mark.parametrize("shape", [(2, 256, 16, 16, 64, 1, 1, 2, 0), (1, 40, 15, 13, 24, 1, 1, 3, 0),
                                   (2, 130, 14, 14, 96, 1, 1, 2, 0)])
@pytest.mark.parametrize("L,G", [(64, 0), (32, 3), (64, 1)])
@pytest.mark.parametrize("partials", [True, False])
def test_bwd_wt_strided_1x1(shape, L, G, partials):
    # without partials, backward-data also runs over the P x Q grid and is
    # scattered into dx (zeros at the pixels no output reads)
    n, c, h, w, k, r, s, st, pd = shape
    d = dfp.make_desc(n, c, h, w, k, r, s, st, pd, chunk_len=L, seg_chunks=G)
    assert dfp.workspace_bytes(d, dfp.BWD_WT) > 0  # the MFMA path (the VALU path needs no workspace)
    run_all(shape, L, G=G, partials=partials)


# Unit-stride 1x1 layers without padding, without partials: both operands as
# digit blocks (channel counts that are not multiples of 64, reductions that
# end mid-chunk, one to many segments; the strided shape takes the same
# kernel on its subsampled input).  0 ulp against the oracle.
# P*Q a multiple of 16 (the last four shapes) reads the INT16 tensors directly.
@pytest.mark.parametrize("shape", [(2, 96, 7, 7, 130, 1, 1, 1, 0), (1, 64, 14, 14, 64, 1, 1, 1, 0),
                                   (3, 40, 5, 9, 24, 1, 1, 1, 0), (2, 256, 16, 16, 64, 1, 1, 2, 0),
                                   (2, 96, 8, 8, 130, 1, 1, 1, 0), (3, 40, 4, 12, 24, 1, 1, 1, 0),
                                   (1, 64, 16, 16, 64, 1, 1, 1, 0)])
@pytest.mark.parametrize("L,G", [(64, 0), (32, 3), (128, 1), (64, 10 ** 6)])
def test_bwd_wt_1x1_digit_blocks(shape, L, G):
    run_all(shape, L, G=G, partials=False)


# Without partials, L = 64 runs the flat-band kernel on the 3x3 shapes here
# (with partials the eight-wave band kernel): segments of one chunk, of an odd
# number of chunks (a last band of one chunk), several bands, one segment per
# layer.
@pytest.mark.parametrize("shape", BAND_SHAPES + [(2, 64, 56, 56, 64, 3, 3, 1, 1)])
@pytest.mark.parametrize("G", [0, 1, 3, 5, 10 ** 6])
def test_bwd_wt_band_no_partials(shape, G):
    run_all(shape, 64, G=G, partials=False)


# Wide rows: the flat-band kernel's widest planes (VGG-16's 224-wide rows,
# halo 240) and width 160 (halo 240 too); width 240 runs the eight-wave band
# kernel's one-workgroup-per-CU build (buffers beyond two workgroups' share of
# LDS), 256 and 320 the general kernel (a band of 16 channels no longer fits).
@pytest.mark.parametrize("shape", [(1, 16, 4, 224, 32, 3, 3, 1, 1), (2, 24, 3, 160, 40, 3, 3, 1, 1),
                                   (1, 16, 4, 240, 32, 3, 3, 1, 1), (1, 16, 4, 256, 32, 3, 3, 1, 1),
                                   (1, 8, 2, 320, 24, 3, 3, 1, 1)])
@pytest.mark.parametrize("G", [0, 1, 3, 10 ** 6])
def test_bwd_wt_band_wide_rows(shape, G):
    run_all(shape, 64, G=G, partials=False)


# Shapes with runs that are not 3x3 same-padding layers, without partials at
# L = 64: the eight-wave band kernel with runs of 8 (output width 16) and of 4
# (widths 28 and 12), 1x3 filters with column padding only and a 3x1 filter
# without padding.
@pytest.mark.parametrize("shape,pad_w", [((2, 16, 8, 16, 32, 1, 3, 1, 0), 1), ((8, 24, 6, 28, 40, 1, 3, 1, 0), 1),
                                         ((4, 16, 10, 8, 48, 3, 1, 1, 0), 0), ((4, 32, 8, 12, 20, 1, 3, 1, 0), 1)])
@pytest.mark.parametrize("G", [0, 1, 3, 10 ** 6])
def test_bwd_wt_band_not_flat(shape, pad_w, G):
    run_all(shape, 64, G=G, partials=False, pad_w=pad_w)


# Output widths that are multiples of 4 but not of 8 (ResNet-50's 28 x 28
# layers): 3x3 same-padding layers, so without partials at L = 64 the
# flat-band kernel; Q = 4, two 64-row dy tiles, segments of one chunk to the
# whole reduction.
RUN4_SHAPES = [
    (4, 16, 12, 12, 32, 3, 3, 1, 1),
    (4, 24, 20, 20, 40, 3, 3, 1, 1),
    (4, 64, 28, 28, 64, 3, 3, 1, 1),
    (4, 32, 12, 4, 20, 3, 3, 1, 1),
    (8, 16, 10, 12, 80, 3, 3, 1, 1),
]


@pytest.mark.parametrize("shape", RUN4_SHAPES)
@pytest.mark.parametrize("G", [0, 1, 3, 10 ** 6])
def test_bwd_wt_band_runs_of_4(shape, G):
    n, c, h, w, k, r, s, st, pd = shape
    assert (w % 8) == 4 and (n * h * w) % 64 == 0
    run_all(shape, 64, G=G, partials=False)


# 3x3 layers with unit stride and one pixel of padding on images narrower
# than 16 whose output width is not a multiple of 4 (ResNet-50's 14 x 14 and
# 7 x 7 layers): at L = 64 the flat-band kernel (with partials its
# two-waves-per-SIMD build, which also stores every chunk partial) takes the
# backward-weights (windows over t-ordered input planes, selector-masked at
# image edges).  Ragged column tiles (C*9 not a multiple of 128), fewer than
# 16 channels, ragged dy row tiles, one-column images, width 15 (the widest
# shift), odd widths, and segments of one chunk to the whole reduction.
FLAT_SHAPES = [
    (64, 16, 7, 7, 64, 3, 3, 1, 1),
    (16, 32, 14, 14, 40, 3, 3, 1, 1),
    (64, 8, 7, 7, 16, 3, 3, 1, 1),
    (32, 16, 6, 6, 32, 3, 3, 1, 1),
    (64, 24, 5, 15, 24, 3, 3, 1, 1),
    (64, 16, 8, 1, 32, 3, 3, 1, 1),
    (64, 16, 13, 13, 72, 3, 3, 1, 1),
]


@pytest.mark.parametrize("shape", FLAT_SHAPES)
@pytest.mark.parametrize("G", [0, 1, 3, 10 ** 6])
@pytest.mark.parametrize("partials", [False, True])
def test_bwd_wt_flat_band(shape, G, partials):
    n, c, h, w, k, r, s, st, pd = shape
    assert (w % 4) != 0 and w < 16 and (n * h * w) % 64 == 0
    run_all(shape, 64, G=G, partials=partials)


# Strided backward-data without partials at L = 64 with K a multiple of 64:
# split by output phase into unit-stride problems over the undilated dy (the
# stem's 7x7 stride 2 on C = 3, odd sizes, 3x3 / 5x5 / 4x4 / 2x2 filters,
# stride 3, phases whose only tap is a 1x1 without padding, and a 1x3
# filter whose odd-row phases receive no tap at all).
PHASE_SHAPES = [
    (2, 3, 16, 16, 64, 7, 7, 2, 3),
    (2, 5, 15, 13, 64, 7, 7, 2, 3),
    (2, 16, 14, 14, 64, 3, 3, 2, 1),
    (2, 16, 13, 11, 128, 3, 3, 2, 1),
    (2, 8, 9, 9, 64, 5, 5, 2, 2),
    (2, 4, 10, 10, 64, 3, 3, 3, 1),
    (1, 3, 20, 20, 64, 4, 4, 2, 1),
    (2, 6, 12, 12, 64, 2, 2, 2, 0),
    (2, 8, 12, 12, 64, 1, 3, 2, 0),
]


@pytest.mark.parametrize("shape", PHASE_SHAPES)
def test_bwd_data_phases(shape):
    run_all(shape, 64, partials=False)


# 32-channel blocks with reductions a multiple of 64 at L = 64: the
# four-waves-per-SIMD kernel over the plane layout takes the forward (and the
# backward-data where K is a multiple of 32), across one-chunk reductions
# (T = 64), several 64-row tiles with a ragged last one, the largest resident
# filter (36 blocks), larger filters in phases of at most 36 blocks (the
# chunk sums carried in the output between launches), strides, and fewer
# output pixels than one wave's unit.
W16_SHAPES = [
    (2, 64, 12, 12, 64, 3, 3, 1, 1),
    (2, 64, 16, 16, 128, 3, 3, 2, 1),  # strided: backward-data reads a dilated plane
    (2, 64, 20, 12, 64, 1, 1, 1, 0),   # no padding columns
    (1, 256, 6, 6, 64, 3, 3, 1, 1),    # 72 filter blocks: two phases of 18 chunks
    (1, 512, 4, 5, 96, 3, 3, 1, 1),    # 144 blocks: four phases
    (2, 96, 6, 6, 416, 3, 3, 2, 1),    # 27 chunks: phases of 13 and 14; 416 rows, ragged tile
    (2, 64, 7, 7, 64, 1, 1, 1, 0),
    (1, 64, 13, 13, 200, 3, 3, 1, 1),
    (2, 128, 5, 5, 192, 3, 3, 1, 1),
    (2, 64, 14, 14, 64, 3, 3, 2, 1),
    (2, 64, 14, 14, 128, 1, 1, 2, 0),
    (1, 64, 2, 3, 64, 3, 3, 1, 1),
]


@pytest.mark.parametrize("shape", W16_SHAPES)
@pytest.mark.parametrize("partials", [True, False])
def test_w16_shapes(shape, partials):
    run_all(shape, 64, path=dfp.PATH_MFMA, partials=partials)


# Fewer 32 x 32 output tiles than the chip's wave slots, every phase an even
# number of chunks, no partials: the 16 x 16-tile kernel (ResNet-50's 14 x 14
# and 7 x 7 layers): one to six phases of up to 72 blocks (reductions of 144,
# 216 and 432 blocks), ragged pixel tiles, output channels not a multiple of
# 64 (nor of 16), stride 2 (backward-data of that shape reads a dilated
# plane), 1 x 1 with two and four chunks.
S16_SHAPES = [
    (2, 256, 14, 14, 64, 3, 3, 1, 1),
    (1, 768, 5, 5, 64, 3, 3, 1, 1),
    (1, 512, 7, 7, 96, 3, 3, 1, 1),
    (2, 128, 5, 5, 192, 3, 3, 1, 1),
    (2, 128, 10, 10, 64, 3, 3, 2, 1),
    (2, 128, 8, 8, 256, 1, 1, 1, 0),
    (4, 256, 7, 7, 512, 3, 3, 1, 1),
    (1, 512, 6, 6, 40, 3, 3, 1, 1),
    (1, 1536, 3, 3, 48, 3, 3, 1, 1),
]


@pytest.mark.parametrize("shape", S16_SHAPES)
def test_s16_shapes(shape):
    run_all(shape, 64, path=dfp.PATH_MFMA, partials=False)


# Forward with fewer than 16 input channels and S*C >= 16 (the 7x7 stem's
# C = 3): channel-last digit rows, a lane's 16 indices as at most two byte runs
# merged with byte masks.  S*C = 16 exactly, wide and narrow filters, C = 1,
# strides 1 and 2, output channels not a multiple of 64 (two row tiles),
# reductions ending mid-block (odd block counts: a last chunk of one block).
CL_SHAPES = [
    (2, 3, 20, 20, 64, 7, 7, 2, 3),
    (2, 4, 10, 10, 32, 4, 4, 1, 1),
    (1, 2, 12, 12, 40, 3, 9, 1, 4),
    (3, 1, 30, 30, 16, 5, 16, 1, 2),
    (2, 3, 17, 17, 96, 7, 7, 2, 3),
    (1, 5, 9, 11, 70, 2, 4, 1, 1),
]


# Unit-stride 1x1 layers with many pixels (N*P*Q >= 32768) and short
# reductions (at most 8 blocks): forward and backward-data read the NCHW
# activations through LDS (no plane preparation).  Output channels not a
# multiple of 64, reductions ending mid-block and an odd block count (the
# last band one block), chunk lengths spanning bands.
STAGED_1X1_SHAPES = [
    (8, 64, 64, 64, 96, 1, 1, 1, 0),
    (4, 200, 96, 96, 40, 1, 1, 1, 0),
]


@pytest.mark.parametrize("shape", STAGED_1X1_SHAPES)
@pytest.mark.parametrize("L", [64, 32, 96])
@pytest.mark.parametrize("partials", [True, False])
def test_1x1_staged(shape, L, partials):
    run_all(shape, L, partials=partials)


@pytest.mark.parametrize("shape", CL_SHAPES)
@pytest.mark.parametrize("partials", [True, False])
def test_few_channel_forward(shape, partials):
    n, c, h, w, k, r, s, st, pd = shape
    assert c < 16 and s * c >= 16
    run_all(shape, 64, partials=partials)


@pytest.mark.parametrize("G", [1, 2, 3, 50])
def test_bwd_wt_segments(G):
    run_all((4, 16, 12, 12, 8, 3, 3, 1, 1), 16, G=G)


def test_stochastic_chain_and_downconvert():
    """quantise -> conv -> down-convert, stochastic rounding, both amax routes."""
    res = run_all((2, 16, 14, 14, 32, 3, 3, 1, 1), 16, rounding="stochastic", seed=9)
    for direction, role in ((dfp.FWD, dfp.ROLE_Y), (dfp.BWD_DATA, dfp.ROLE_DX)):
        gl, out, so, ref = res[direction]
        oq, oe, ofl = oracle.quantize(ref, 15, oracle.ROUND_STOCHASTIC, 9, role)
        for sc in (so, None):  # epilogue max, then a fresh max pass
            q, s2 = gl.downconvert(out, role, sc)
            torch.cuda.synchronize()
            assert np.array_equal(q.cpu().numpy(), oq)
            info = dfp.read_scale(s2)
            assert info["exp"] == oe and info["flags"] == ofl
            assert info["amax_bits"] == int((ref.view(np.uint32) & 0x7fffffff).max())


def test_overflow_wraps_like_oracle():
    """All operands at +2^14 (DFP15 max): 8 products reach 2^31 and wrap to -2^31."""
    for L in (7, 8, 9, 64):
        gl = GpuLayer(1, 64, 4, 4, 8, 3, 3, 1, 1, L=L)
        v = np.float32(16383.75 / 8192)  # x = 16383.75 rounds to 2^14 (Es = -13)
        fx = np.full(gl.shape_x, v, np.float32)
        fw = np.full(gl.shape_w, v, np.float32)
        qx, sx = gl.quantize(fx, dfp.ROLE_X)
        qw, sw = gl.quantize(fw, dfp.ROLE_W)
        ox, ex, _ = oracle.quantize(fx, 15)
        ow, ew, _ = oracle.quantize(fw, 15)
        assert int(ox.max()) == 2 ** 14
        g = oracle_geom(gl)
        out, _, parts = gl.conv(dfp.FWD, qx, sx, qw, sw, want_partials=True)
        ref, rparts, ov = oracle.conv(g, oracle.FWD, ox, ow, ex + ew, L, want_partials=True)
        torch.cuda.synchronize()
        assert np.array_equal(parts.cpu().numpy(), rparts)
        assert np.array_equal(out.cpu().numpy(), ref)
        if L >= 8:
            assert ov > 0


def test_p16_three_products_overflow():
    gl = GpuLayer(1, 3, 1, 1, 1, 1, 1, L=3, bits=16)
    v = np.full(gl.shape_x, np.float32(32767.0 / 16384.0))
    qx, sx = gl.quantize(v, dfp.ROLE_X)
    qw, sw = gl.quantize(v.reshape(gl.shape_w), dfp.ROLE_W)
    out, _, parts = gl.conv(dfp.FWD, qx, sx, qw, sw, want_partials=True)
    torch.cuda.synchronize()
    assert int(qx.cpu().numpy().reshape(-1)[0]) == 32767
    assert int(parts.cpu().numpy()[0, 0]) == -1073938429


def test_scale_extremes():
    """Ea + Eb far outside FP32: outputs overflow to inf (OUTPUT_INF) or land in
    the subnormal range with a single rounding."""
    for sc_x, sc_w in ((3e38, 3e38), (1e-30, 1e-30), (2e-20, 1e-19)):
        gl = GpuLayer(1, 8, 5, 5, 4, 3, 3, 1, 1, L=16)
        rng = np.random.default_rng(3)
        x = (rng.standard_normal(gl.shape_x) * sc_x).astype(np.float32)
        w = (rng.standard_normal(gl.shape_w) * sc_w).astype(np.float32)
        x = np.clip(x, -3e38, 3e38)
        w = np.clip(w, -3e38, 3e38)
        qx, sx = gl.quantize(x, dfp.ROLE_X)
        qw, sw = gl.quantize(w, dfp.ROLE_W)
        ox, ex, _ = oracle.quantize(x, 15)
        ow, ew, _ = oracle.quantize(w, 15)
        out, so, _ = gl.conv(dfp.FWD, qx, sx, qw, sw)
        ref, _, _ = oracle.conv(oracle_geom(gl), oracle.FWD, ox, ow, ex + ew, 16)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
        flags = dfp.read_scale(so)["flags"]
        assert bool(flags & dfp.FLAG_OUTPUT_INF) == bool(np.isinf(ref).any())


def test_layer16x32_full_chain():
    """The 2x16x14x14, 16->32 3x3 layer of the workload list (seed 0, nearest,
    L = 16): every stage bit-exact, both down-converts."""
    from paper_1802_00930_amd.workloads import WORKLOADS, layer_inputs
    wl = WORKLOADS["layer16x32"]
    layer, x, w, dy = layer_inputs(wl, 0)
    gl = GpuLayer(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad, L=16)
    qx, sx = gl.quantize(x, dfp.ROLE_X)
    qw, sw = gl.quantize(w, dfp.ROLE_W)
    qdy, sdy = gl.quantize(dy, dfp.ROLE_DY)
    ox, ex, _ = oracle.quantize(x, 15, 0, 0, 0)
    ow, ew, _ = oracle.quantize(w, 15, 0, 0, 1)
    ody, edy, _ = oracle.quantize(dy, 15, 0, 0, 2)
    g = oracle_geom(gl)
    y, sy, py = gl.conv(dfp.FWD, qx, sx, qw, sw, want_partials=True)
    dx, sdx, pdx = gl.conv(dfp.BWD_DATA, qdy, sdy, qw, sw, want_partials=True)
    dw, _, pdw = gl.conv(dfp.BWD_WT, qx, sx, qdy, sdy, want_partials=True)
    qy, sqy = gl.downconvert(y, dfp.ROLE_Y, sy)
    qdx, sqdx = gl.downconvert(dx, dfp.ROLE_DX, sdx)
    oy, opy, _ = oracle.conv(g, oracle.FWD, ox, ow, ex + ew, 16, want_partials=True)
    odx, opdx, _ = oracle.conv(g, oracle.BWD_DATA, ody, ow, edy + ew, 16, want_partials=True)
    odw, opdw, _ = oracle.conv(g, oracle.BWD_WT, ox, ody, ex + edy, 16, want_partials=True)
    oqy, eqy, _ = oracle.quantize(oy, 15, 0, 0, 3)
    oqdx, eqdx, _ = oracle.quantize(odx, 15, 0, 0, 4)
    torch.cuda.synchronize()
    assert np.array_equal(qx.cpu().numpy(), ox) and dfp.read_scale(sx)["exp"] == ex
    assert np.array_equal(qw.cpu().numpy(), ow) and dfp.read_scale(sw)["exp"] == ew
    assert np.array_equal(qdy.cpu().numpy(), ody) and dfp.read_scale(sdy)["exp"] == edy
    for got, ref in ((py, opy), (pdx, opdx), (pdw, opdw)):
        assert np.array_equal(got.cpu().numpy(), ref)
    for got, ref in ((y, oy), (dx, odx), (dw, odw)):
        assert np.array_equal(got.cpu().numpy(), ref)
    assert np.array_equal(qy.cpu().numpy(), oqy) and dfp.read_scale(sqy)["exp"] == eqy
    assert np.array_equal(qdx.cpu().numpy(), oqdx) and dfp.read_scale(sqdx)["exp"] == eqdx


def test_deterministic():
    shape = (2, 64, 10, 10, 64, 3, 3, 1, 1)
    gl = GpuLayer(*shape, L=64)
    rng = np.random.default_rng(1)
    qx, sx = gl.quantize(rng.standard_normal(gl.shape_x).astype(np.float32), dfp.ROLE_X)
    qdy, sdy = gl.quantize(rng.standard_normal(gl.shape_y).astype(np.float32), dfp.ROLE_DY)
    qw, sw = gl.quantize(rng.standard_normal(gl.shape_w).astype(np.float32), dfp.ROLE_W)
    for direction, a, sa, b, sb in ((dfp.FWD, qx, sx, qw, sw), (dfp.BWD_DATA, qdy, sdy, qw, sw),
                                    (dfp.BWD_WT, qx, sx, qdy, sdy)):
        o1, _, _ = gl.conv(direction, a, sa, b, sb)
        o2, _, _ = gl.conv(direction, a, sa, b, sb)
        torch.cuda.synchronize()
        assert torch.equal(o1.view(torch.int32), o2.view(torch.int32))

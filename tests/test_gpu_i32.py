"""GPU parity of the DFP-32 outputs and the integer down-convert (Eq. 6)
against the CPU oracle: the single-chunk INT32 convolutions bit-exact against
the oracle's one chunk partial, their scales (exp = Ea + Eb, max |i|) exact,
and the integer down-convert bit-exact in every rounding mode, at both
precisions, with and without a precomputed max, across its degenerate cases
(an all-zero tensor, -2^31, a max below 2^(P-2) so the shift is to the left,
an exponent that clamps at -128, ragged and tiny lengths, ties)."""
import zlib

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, GpuLayer, note, oracle_geom, to_dev
from paper_1802_00930_amd import dfp

pytestmark = pytest.mark.gpu

SHAPES = [
    # n, c, h, w, k, r, s, stride, pad
    (2, 16, 14, 14, 32, 3, 3, 1, 1),
    (2, 3, 9, 8, 4, 3, 3, 1, 1),
    (2, 4, 10, 9, 5, 3, 3, 2, 1),
    (1, 3, 23, 23, 8, 7, 7, 2, 3),
    (3, 64, 9, 11, 40, 3, 3, 1, 1),
    (2, 96, 7, 7, 130, 1, 1, 1, 0),
    (1, 70, 12, 12, 33, 3, 3, 2, 1),
    (2, 512, 7, 7, 64, 3, 3, 1, 1),  # 4608 products per forward output: INT32 sums wrap
    # reductions that are multiples of 64 with 4..18 blocks of 32 (the persistent kernel)
    (2, 64, 10, 10, 64, 3, 3, 1, 1),
    (1, 128, 8, 8, 192, 1, 1, 1, 0),
    (2, 64, 13, 11, 72, 3, 3, 2, 1),
    (3, 128, 5, 7, 64, 3, 3, 1, 1),
]


def scale_tensor(exp, amax=0):
    return torch.tensor([amax & 0xffffffff if amax < 2 ** 31 else amax - 2 ** 32, exp, 0, 0], dtype=torch.int32,
                        device=DEV)


def red_len(shape, direction):
    n, c, h, w, k, r, s, _, _ = shape
    return (c if direction == dfp.FWD else k) * r * s


def conv_i32(gl, direction, a, sa, b, sb):
    shape = gl.shape_y if direction == dfp.FWD else gl.shape_x
    out = torch.full(shape, 0x5a5a5a5a, dtype=torch.int32, device=DEV)
    so = scale_tensor(77, 0x12345)  # the call must overwrite every field it defines
    ws = dfp.alloc_workspace(gl.d, direction, DEV)
    if direction == dfp.FWD:
        dfp.dfp_conv_fwd_i32(gl.d, a, sa, b, sb, out, so, ws)
    else:
        dfp.dfp_conv_bwd_data_i32(gl.d, a, sa, b, sb, out, so, ws)
    return out, so


def check_conv_i32(shape, path, extra, full_range, seed=0):
    n, c, h, w, k, r, s, st, pd = shape
    rng = np.random.default_rng([seed, n, c, h, w, k, r, s, st, pd, path, extra])
    lim = 32767 if full_range else 16384
    for direction in (dfp.FWD, dfp.BWD_DATA):
        L = red_len(shape, direction) + extra
        gl = GpuLayer(n, c, h, w, k, r, s, st, pd, L=L, path=path)
        g = oracle_geom(gl)
        a_shape = gl.shape_x if direction == dfp.FWD else gl.shape_y
        a = rng.integers(-lim, lim + 1, a_shape).astype(np.int16)
        b = rng.integers(-lim, lim + 1, gl.shape_w).astype(np.int16)
        ea, eb = int(rng.integers(-20, -5)), int(rng.integers(-20, -5))
        note("conv_i32 shape=%s dir=%d path=%d L=%d full=%d" % (shape, direction, path, L, full_range))
        out, so = conv_i32(gl, direction, to_dev(a), scale_tensor(ea), to_dev(b), scale_tensor(eb))
        _, rparts, _ = oracle.conv(g, direction, a, b, ea + eb, L, 1, want_partials=True)
        torch.cuda.synchronize()
        assert rparts.shape[0] == 1
        got = out.cpu().numpy().reshape(-1)
        ref = rparts[0]
        bad = np.nonzero(got != ref)[0]
        assert bad.size == 0, "dir %d: %d outputs differ, first %s gpu=%s ref=%s" % (
            direction, bad.size, bad[:4], got[bad[:4]], ref[bad[:4]])
        sc = dfp.read_scale(so)
        assert sc["exp"] == ea + eb
        assert sc["amax_bits"] == int(np.abs(ref.astype(np.int64)).max())
        assert sc["flags"] == 0


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("path", [dfp.PATH_MFMA, dfp.PATH_VALU])
def test_conv_i32_matches_oracle(shape, path):
    # P = 15 operands (|i| <= 2^14) on both paths; the full INT16 range on the
    # VALU path, which also serves P = 16
    check_conv_i32(shape, path, extra=0, full_range=False)
    if path == dfp.PATH_VALU:
        check_conv_i32(shape, path, extra=0, full_range=True, seed=1)


@pytest.mark.parametrize("shape", SHAPES[:3] + SHAPES[5:6])
def test_conv_i32_longer_chunk_and_dfp_range(shape):
    # a chunk longer than the reduction is the same single chunk; inputs in the
    # range the quantiser produces
    check_conv_i32(shape, dfp.PATH_AUTO, extra=1000, full_range=False, seed=3)


def test_conv_i32_equals_fp32_path_single_chunk():
    """With one chunk the FP32-output call returns 2^e * float(I) for the same
    INT32 I (Alg. 2 with J = 1); both outputs are taken from the GPU."""
    shape = (2, 64, 12, 12, 64, 3, 3, 1, 1)
    n, c, h, w, k, r, s, st, pd = shape
    rng = np.random.default_rng(11)
    gl = GpuLayer(n, c, h, w, k, r, s, st, pd, L=c * r * s)
    x = to_dev(rng.integers(-16384, 16385, gl.shape_x).astype(np.int16))
    wt = to_dev(rng.integers(-16384, 16385, gl.shape_w).astype(np.int16))
    sx, sw = scale_tensor(-13), scale_tensor(-17)
    yi, syi = conv_i32(gl, dfp.FWD, x, sx, wt, sw)
    yf, syf, _ = gl.conv(dfp.FWD, x, sx, wt, sw)
    torch.cuda.synchronize()
    expect = np.ldexp(yi.cpu().numpy().astype(np.float32), -30).astype(np.float32)
    assert np.array_equal(yf.cpu().numpy(), expect)


# --------------------------------------------------------------------------
# integer down-convert
# --------------------------------------------------------------------------
def downconvert_case(name, rng, bits):
    """(int32 values, exponent of the DFP-32 input)."""
    if name == "wide":
        return rng.integers(-2 ** 31 + 1, 2 ** 31, 100003).astype(np.int32), -20
    if name == "int_min":
        v = rng.integers(-2 ** 20, 2 ** 20, 10007).astype(np.int32)
        v[5000] = -2 ** 31
        return v, -40
    if name == "small_max":  # max |i| < 2^(P-2): exact left shift
        return rng.integers(-200, 201, 4099).astype(np.int32), 3
    if name == "zero":
        return np.zeros(4101, dtype=np.int32), -7
    if name == "clamp":  # E_in + Rs < -128
        return rng.integers(-2 ** 20, 2 ** 20, 5003).astype(np.int32), -140
    if name == "clamp_far":  # the clamp pushes the shift to about 36 bits (past the 32-bit fraction)
        return rng.integers(-2 ** 30, 2 ** 30, 3001).astype(np.int32), -164
    if name == "ties":  # max at bit 30, so Rs = 30 - (P-2); every value an exact half step
        rs = 30 - (bits - 2)
        v = (rng.integers(-2 ** 12, 2 ** 12, 8191).astype(np.int64) << rs) + (1 << (rs - 1))
        v[0] = 2 ** 30 + (1 << (rs - 1))
        return v.astype(np.int32), 0
    if name == "tiny":
        return np.array([-3], dtype=np.int32), 1
    if name == "three":
        return np.array([2 ** 20 + 1, -5, 7], dtype=np.int32), -2
    if name == "big":  # several amax partial blocks, ragged tail
        return rng.integers(-2 ** 27, 2 ** 27, 3 * 2 ** 20 + 5).astype(np.int32), -30
    raise KeyError(name)


CASES = ["wide", "int_min", "small_max", "zero", "clamp", "clamp_far", "ties", "tiny", "three", "big"]


def run_downconvert(vals, e_in, bits, rounding, ready, role, seed):
    n = vals.size
    d = dfp.make_desc(1, 1, 1, n, 1, 1, 1, bits=bits, rounding=rounding, seed=seed)
    src = to_dev(vals)
    mx = int(np.abs(vals.astype(np.int64)).max())
    sin = scale_tensor(e_in, mx if ready else 0x3f00)  # with ready = 0 the max must be recomputed
    dst = torch.full((n,), 0x7777, dtype=torch.int16, device=DEV)
    sout = scale_tensor(99, 0x55)
    dfp.dfp_downconvert_i32(d, role, src, sin, dst, sout, amax_ready=ready)
    torch.cuda.synchronize()
    return dst.cpu().numpy(), dfp.read_scale(sout), mx


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("rounding", ["nearest", "biased", "stochastic", "down"])
@pytest.mark.parametrize("bits", [15, 16])
@pytest.mark.parametrize("ready", [0, 1])
def test_downconvert_i32_matches_oracle(case, rounding, bits, ready):
    rng = np.random.default_rng(zlib.crc32(("%s/%d" % (case, bits)).encode()))
    vals, e_in = downconvert_case(case, rng, bits)
    seed = 0x0123456789 if rounding == "stochastic" else 0
    role = dfp.ROLE_Y if ready else dfp.ROLE_DX
    note("downconvert_i32 case=%s rounding=%s bits=%d ready=%d n=%d" % (case, rounding, bits, ready, vals.size))
    got, sc, mx = run_downconvert(vals, e_in, bits, rounding, ready, role, seed)
    ref, e_ref, f_ref = oracle.downconvert_i32(vals, e_in, bits, oracle.ROUNDING[rounding], seed, role)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, "%d differ, first %s gpu=%s ref=%s" % (bad.size, bad[:4], got[bad[:4]], ref[bad[:4]])
    assert sc["exp"] == e_ref
    assert sc["flags"] == f_ref
    assert sc["amax_bits"] == mx


def test_downconvert_i32_roles_draw_different_streams():
    rng = np.random.default_rng(5)
    vals = rng.integers(-2 ** 28, 2 ** 28, 65536).astype(np.int32)
    a, _, _ = run_downconvert(vals, -10, 15, "stochastic", 1, dfp.ROLE_Y, 42)
    b, _, _ = run_downconvert(vals, -10, 15, "stochastic", 1, dfp.ROLE_DX, 42)
    rb, _, _ = oracle.downconvert_i32(vals, -10, 15, oracle.ROUNDING["stochastic"], 42, oracle.ROLE_DX)
    assert np.array_equal(b, rb)
    assert np.count_nonzero(a != b) > 1000


@pytest.mark.parametrize("rounding", ["nearest", "stochastic"])
@pytest.mark.parametrize("bits", [15, 16])
def test_chain_quantize_conv_i32_downconvert(rounding, bits):
    """FP32 tensors -> DFP (Eq. 2) -> single-chunk DFP-32 forward and
    backward-data -> integer down-convert with the epilogue's max (Eq. 6),
    every stage on the GPU against the same stages of the oracle."""
    shape = (2, 32, 15, 13, 48, 3, 3, 1, 1)
    n, c, h, w, k, r, s, st, pd = shape
    rng = np.random.default_rng(bits)
    seed = 7
    for direction in (dfp.FWD, dfp.BWD_DATA):
        gl = GpuLayer(n, c, h, w, k, r, s, st, pd, L=red_len(shape, direction), bits=bits, rounding=rounding,
                      seed=seed)
        g = oracle_geom(gl)
        rnd = oracle.ROUNDING[rounding]
        a_role = dfp.ROLE_X if direction == dfp.FWD else dfp.ROLE_DY
        a_f = rng.standard_normal(gl.shape_x if direction == dfp.FWD else gl.shape_y).astype(np.float32)
        w_f = (rng.standard_normal(gl.shape_w) * 0.05).astype(np.float32)
        qa, sa = gl.quantize(a_f, a_role)
        qw, sw = gl.quantize(w_f, dfp.ROLE_W)
        oa, ea, _ = oracle.quantize(a_f, bits, rnd, seed, a_role)
        ow, ew, _ = oracle.quantize(w_f, bits, rnd, seed, dfp.ROLE_W)
        out, so = conv_i32(gl, direction, qa, sa, qw, sw)
        role = dfp.ROLE_Y if direction == dfp.FWD else dfp.ROLE_DX
        q = torch.empty(out.shape, dtype=torch.int16, device=DEV)
        sq = dfp.new_scale(DEV)
        dfp.dfp_downconvert_i32(gl.d, role, out, so, q, sq, amax_ready=True)
        _, rparts, _ = oracle.conv(g, direction, oa, ow, ea + ew, gl.d.chunk_len, 1, want_partials=True)
        rq, re, rf = oracle.downconvert_i32(rparts[0], ea + ew, bits, rnd, seed, role)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().reshape(-1), rparts[0])
        assert np.array_equal(q.cpu().numpy().reshape(-1), rq)
        sc = dfp.read_scale(sq)
        assert (sc["exp"], sc["flags"]) == (re, rf)

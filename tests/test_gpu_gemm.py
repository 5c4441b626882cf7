"""GPU parity of the DFP16 GEMM against the CPU oracle: every INT32 chunk
partial bit-exact, FP32 outputs within 1e-6 relative (0 ulp expected), the
epilogue max exact, on both product paths, all four transpose settings,
ragged sizes and masked chunk lengths; the flat quantise / down-convert; and a
fully connected layer (forward, backward-data, backward-weights) end to end.
Large products are checked at sampled rows and columns, computed by the oracle
on the corresponding rows of opA and columns of opB."""
import zlib

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, assert_fp32_close, note, to_dev, ulp_diff
from paper_1802_00930_amd import dfp

pytestmark = pytest.mark.gpu

TRANS = [(False, False), (False, True), (True, False), (True, True)]


def scale_tensor(exp):
    return torch.tensor([0, exp, 0, 0], dtype=torch.int32, device=DEV)


def operands(m, n, k, ta, tb, lim, seed):
    rng = np.random.default_rng(seed)
    op_a = rng.integers(-lim, lim + 1, (m, k)).astype(np.int16)
    op_b = rng.integers(-lim, lim + 1, (k, n)).astype(np.int16)
    a = np.ascontiguousarray(op_a.T if ta else op_a)
    b = np.ascontiguousarray(op_b.T if tb else op_b)
    return op_a, op_b, a, b


def run_gemm(m, n, k, ta, tb, L, path=dfp.PATH_AUTO, bits=15, ea=-14, eb=-15, a=None, b=None, partials=True,
             sa=None, sb=None):
    d = dfp.make_gemm_desc(m, n, k, ta, tb, chunk_len=L, bits=bits, path=path)
    out = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
    sd = torch.tensor([123, 7, 9, 0], dtype=torch.int32, device=DEV)  # must be cleared by the call
    ws = dfp.alloc_gemm_workspace(d, DEV)
    parts = None
    if partials:
        parts = torch.full((dfp.gemm_num_chunks(d), m * n), 0x5a5a5a5a, dtype=torch.int32, device=DEV)
    dfp.dfp_gemm(d, a, scale_tensor(ea) if sa is None else sa, b, scale_tensor(eb) if sb is None else sb, out, sd,
                 ws, parts)
    return out, sd, parts


def check(m, n, k, ta, tb, L, path=dfp.PATH_AUTO, bits=15, seed=0):
    lim = 16384 if bits == 15 else 32767
    op_a, op_b, a, b = operands(m, n, k, ta, tb, lim, [seed, m, n, k, ta, tb, L, path, bits])
    note("gemm m=%d n=%d k=%d ta=%d tb=%d L=%d path=%d bits=%d" % (m, n, k, ta, tb, L, path, bits))
    out, sd, parts = run_gemm(m, n, k, ta, tb, L, path, bits, a=to_dev(a), b=to_dev(b))
    ref, rparts, _ = oracle.gemm(a, b, -29, L, ta, tb, want_partials=True)
    torch.cuda.synchronize()
    gp = parts.cpu().numpy()
    bad = np.argwhere(gp != rparts)
    assert bad.size == 0, "partials differ at %s" % bad[:5]
    got = out.cpu().numpy()
    assert_fp32_close(got, ref, "gemm")
    assert ulp_diff(got, ref) == 0
    s = dfp.read_scale(sd)
    assert s["amax_bits"] == int((ref.view(np.uint32) & 0x7fffffff).max())
    assert s["flags"] == oracle.output_flags(ref)


SHAPES = [
    (1, 1, 1),
    (13, 37, 150),
    (64, 64, 128),      # 4 blocks of 32, k a multiple of 64: persistent kernel at L = 64
    (130, 257, 96),
    (200, 300, 640),    # 20 blocks: the largest resident filter
    (5, 700, 33),
    (300, 9, 1000),     # k = 1000: a ragged last block
    (64, 1000, 2048),   # ResNet-50's FC layer forward (batch 64)
]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("ta,tb", TRANS)
def test_gemm_matches_oracle(shape, ta, tb):
    m, n, k = shape
    for L in (64, 32):
        check(m, n, k, ta, tb, L)


@pytest.mark.parametrize("L", [1, 5, 16, 96, 10 ** 6])
@pytest.mark.parametrize("path", [dfp.PATH_MFMA, dfp.PATH_VALU])
def test_gemm_chunk_lengths_and_paths(L, path):
    for m, n, k in ((13, 37, 150), (130, 66, 300)):
        check(m, n, k, False, True, L, path)
        check(m, n, k, True, False, L, path)


@pytest.mark.parametrize("ta,tb", TRANS)
def test_gemm_p16_full_range(ta, tb):
    check(37, 41, 300, ta, tb, 64, dfp.PATH_AUTO, bits=16)


def test_gemm_wraps_like_the_oracle():
    # full-range DFP15 operands over a 2000-long single chunk: most partials wrap
    m, n, k = 33, 65, 2000
    op_a, op_b, a, b = operands(m, n, k, False, False, 16384, 9)
    out, _, parts = run_gemm(m, n, k, False, False, 2000, a=to_dev(a), b=to_dev(b))
    ref, rparts, wrapped = oracle.gemm(a, b, -29, 2000, want_partials=True)
    torch.cuda.synchronize()
    assert wrapped > 0
    assert np.array_equal(parts.cpu().numpy(), rparts)
    assert ulp_diff(out.cpu().numpy(), ref) == 0


@pytest.mark.parametrize("shape,ta,tb", [((2048, 2048, 2048), False, True), ((4096, 1024, 3072), True, False),
                                         ((1000, 4096, 64), True, False)])
def test_gemm_large_sampled(shape, ta, tb):
    m, n, k = shape
    op_a, op_b, a, b = operands(m, n, k, ta, tb, 16384, 5)
    note("gemm large %s ta=%d tb=%d" % (shape, ta, tb))
    out, sd, _ = run_gemm(m, n, k, ta, tb, 64, a=to_dev(a), b=to_dev(b), partials=False)
    rng = np.random.default_rng(zlib.crc32(repr(shape).encode()))
    rows = np.unique(np.concatenate([rng.integers(0, m, 24), [0, m - 1]]))
    cols = np.unique(np.concatenate([rng.integers(0, n, 24), [0, n - 1]]))
    ref, _, _ = oracle.gemm(op_a[rows], op_b[:, cols], -29, 64)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert ulp_diff(got[np.ix_(rows, cols)], ref) == 0
    s = dfp.read_scale(sd)
    assert s["amax_bits"] == int((got.view(np.uint32) & 0x7fffffff).max())


@pytest.mark.parametrize("rounding", ["nearest", "stochastic"])
@pytest.mark.parametrize("bits", [15, 16])
def test_flat_quantize_and_downconvert(rounding, bits):
    rng = np.random.default_rng(bits)
    for n in (1, 7, 4099, 2 ** 20 + 3):
        f = (rng.standard_normal(n) * 3.0).astype(np.float32)
        for role in (dfp.ROLE_X, dfp.ROLE_DX):
            t = to_dev(f)
            q = torch.empty(n, dtype=torch.int16, device=DEV)
            sc = dfp.new_scale(DEV)
            dfp.dfp_quantize_tensor(bits, rounding, 77, role, t, q, sc)
            q2 = torch.empty(n, dtype=torch.int16, device=DEV)
            sc2 = dfp.new_scale(DEV)
            dfp.dfp_downconvert_tensor(bits, rounding, 77, role, t, q2, sc2)
            ref, e, fl = oracle.quantize(f, bits, oracle.ROUNDING[rounding], 77, role)
            torch.cuda.synchronize()
            for qq, ss in ((q, sc), (q2, sc2)):
                assert np.array_equal(qq.cpu().numpy(), ref)
                s = dfp.read_scale(ss)
                assert (s["exp"], s["flags"]) == (e, fl)


@pytest.mark.parametrize("rounding", ["nearest", "stochastic"])
def test_fully_connected_layer_end_to_end(rounding):
    """ResNet-50's FC layer (2048 -> 1000, batch 64): FP32 x, W, dy quantised
    on the GPU, forward y = x W^T, backward-data dx = dy W, backward-weights
    dW = dy^T x as GEMMs at L = 64, y and dx down-converted with the epilogue
    max; every stage against the oracle."""
    batch, fin, fout, L, seed = 64, 2048, 1000, 64, 3
    rng = np.random.default_rng(4)
    x = np.maximum(rng.standard_normal((batch, fin)), 0).astype(np.float32)
    w = (rng.standard_normal((fout, fin)) * np.sqrt(1.0 / fin)).astype(np.float32)
    dy = (rng.standard_normal((batch, fout)) * 1e-3).astype(np.float32)
    rnd = oracle.ROUNDING[rounding]
    qs = {}
    for name, f, role in (("x", x, dfp.ROLE_X), ("w", w, dfp.ROLE_W), ("dy", dy, dfp.ROLE_DY)):
        q = torch.empty(f.shape, dtype=torch.int16, device=DEV)
        sc = dfp.new_scale(DEV)
        dfp.dfp_quantize_tensor(15, rounding, seed, role, to_dev(f), q, sc)
        oq, oe, _ = oracle.quantize(f, 15, rnd, seed, role)
        torch.cuda.synchronize()
        assert np.array_equal(q.cpu().numpy(), oq)
        assert dfp.read_scale(sc)["exp"] == oe
        qs[name] = (q, sc, oq, oe)
    (qx, sx, ox, ex), (qw, sw, ow, ew), (qdy, sdy, ody, edy) = qs["x"], qs["w"], qs["dy"]
    cases = (("fwd", batch, fout, fin, False, True, qx, sx, qw, sw, ox, ow, ex + ew, dfp.ROLE_Y),
             ("bwd-data", batch, fin, fout, False, False, qdy, sdy, qw, sw, ody, ow, edy + ew, dfp.ROLE_DX),
             ("bwd-wt", fout, fin, batch, True, False, qdy, sdy, qx, sx, ody, ox, edy + ex, None))
    for name, m, n, k, ta, tb, a, sa, b, sb, oa, ob, e, role in cases:
        note("fc %s" % name)
        out, sd, parts = run_gemm(m, n, k, ta, tb, L, a=a, b=b, sa=sa, sb=sb)
        ref, rparts, _ = oracle.gemm(oa, ob, e, L, ta, tb, want_partials=True)
        torch.cuda.synchronize()
        assert np.array_equal(parts.cpu().numpy(), rparts), name
        assert ulp_diff(out.cpu().numpy(), ref) == 0, name
        if role is not None:
            q = torch.empty((m, n), dtype=torch.int16, device=DEV)
            dfp.dfp_downconvert_tensor(15, rounding, seed, role, out, q, sd, amax_ready=True)
            rq, re, _ = oracle.quantize(ref, 15, rnd, seed, role)
            torch.cuda.synchronize()
            assert np.array_equal(q.cpu().numpy(), rq), name
            assert dfp.read_scale(sd)["exp"] == re

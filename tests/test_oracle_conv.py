"""Pins for the oracle's chunked INT16 convolutions (Alg. 2, Sec. 4.3, Eq. 4).

The oracle walks each output's reduction one product at a time.  These tests
hold it against things other than itself:
  * a vectorised int64 brute-force direct convolution (padding by slicing),
  * torch's float64 conv2d / conv2d_input / conv2d_weight on small integers,
    where every chunked FP32 sum is exact (a special case that reduces to the
    library routine), which pins layout, stride, padding and transposition,
  * the exact adjoint identities between the three directions,
  * the overflow figures of Sec. 4.3 and the DFP15 wrap at L = 8,
  * one-hot inputs that land a single product in a known chunk (pins the
    canonical reduction order), and the recursive-summation error bound.
"""
import itertools

import numpy as np
import pytest
import torch

# ------------------------------------------------------------ helpers -----


def brute_fwd(x, w, stride, pad):
    """Exact int64 direct convolution, vectorised over (n, k, p, q)."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    P = (H + 2 * pad - R) // stride + 1
    Q = (W + 2 * pad - S) // stride + 1
    xp = np.zeros((N, C, H + 2 * pad, W + 2 * pad), dtype=np.int64)
    xp[:, :, pad:pad + H, pad:pad + W] = x
    y = np.zeros((N, K, P, Q), dtype=np.int64)
    for r in range(R):
        for s in range(S):
            patch = xp[:, :, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride]
            y += np.einsum("nchw,kc->nkhw", patch, w[:, :, r, s].astype(np.int64))
    return y


def brute_bwd_data(dy, w, H, W, stride, pad):
    N, K, P, Q = dy.shape
    _, C, R, S = w.shape
    dxp = np.zeros((N, C, H + 2 * pad + stride, W + 2 * pad + stride), dtype=np.int64)
    for r in range(R):
        for s in range(S):
            contrib = np.einsum("nkhw,kc->nchw", dy.astype(np.int64), w[:, :, r, s].astype(np.int64))
            dxp[:, :, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride] += contrib
    return dxp[:, :, pad:pad + H, pad:pad + W]


def brute_bwd_wt(x, dy, R, S, stride, pad):
    N, C, H, W = x.shape
    _, K, P, Q = dy.shape
    xp = np.zeros((N, C, H + 2 * pad + stride, W + 2 * pad + stride), dtype=np.int64)
    xp[:, :, pad:pad + H, pad:pad + W] = x
    dw = np.zeros((K, C, R, S), dtype=np.int64)
    for r in range(R):
        for s in range(S):
            patch = xp[:, :, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride]
            dw[:, :, r, s] = np.einsum("nchw,nkhw->kc", patch, dy.astype(np.int64))
    return dw


def wrap32(v):
    return ((np.asarray(v, dtype=np.int64) + 2 ** 31) % 2 ** 32) - 2 ** 31


SHAPES = [
    # n, c, h, w, k, r, s, stride, pad
    (2, 3, 9, 8, 4, 3, 3, 1, 1),
    (1, 5, 7, 7, 3, 1, 1, 1, 0),
    (2, 4, 10, 9, 5, 3, 3, 2, 1),
    (1, 3, 11, 11, 2, 7, 7, 2, 3),
    (2, 8, 6, 6, 6, 1, 1, 2, 0),
    (1, 2, 5, 6, 3, 3, 2, 1, 0),
    (1, 6, 4, 4, 2, 3, 3, 3, 2),
]


def _rand_pair(rng, g, amp):
    P = (g.h + 2 * g.pad_h - g.r) // g.stride_h + 1
    Q = (g.w + 2 * g.pad_w - g.s) // g.stride_w + 1
    x = rng.integers(-amp, amp + 1, (g.n, g.c, g.h, g.w)).astype(np.int16)
    w = rng.integers(-amp, amp + 1, (g.k, g.c, g.r, g.s)).astype(np.int16)
    dy = rng.integers(-amp, amp + 1, (g.n, g.k, P, Q)).astype(np.int16)
    return x, w, dy


# --------------------------------------------------- brute-force int64 ----
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("L", [1, 3, 8, 16, 1000])
def test_partials_sum_to_exact(orc, shape, L):
    g = orc.geom(*shape)
    rng = np.random.default_rng(hash((shape, L)) % 2 ** 32)
    x, w, dy = _rand_pair(rng, g, 2 ** 14)
    cases = [
        (orc.FWD, x, w, brute_fwd(x, w, g.stride_h, g.pad_h)),
        (orc.BWD_DATA, dy, w, brute_bwd_data(dy, w, g.h, g.w, g.stride_h, g.pad_h)),
        (orc.BWD_WT, x, dy, brute_bwd_wt(x, dy, g.r, g.s, g.stride_h, g.pad_h)),
    ]
    for d, a, b, exact in cases:
        out, parts, ov = orc.conv(g, d, a, b, 0, L, want_partials=True)
        assert parts.shape[0] == orc.num_chunks(g, d, L)
        total = parts.astype(np.int64).sum(axis=0)
        assert np.array_equal(wrap32(total), wrap32(exact.reshape(-1)))
        if L <= 3:  # at most 3 * 2^28 < 2^31: nothing can wrap, partial sum is exact
            assert ov == 0 and np.array_equal(total, exact.reshape(-1))


# ----------------------------------------------- torch float64 library ----
@pytest.mark.parametrize("shape", SHAPES)
def test_single_chunk_equals_torch(orc, shape):
    """One chunk (L >= T), exponent 0, small integers: the method computes the
    exact convolution, so it must equal torch's float64 convolutions."""
    g = orc.geom(*shape)
    rng = np.random.default_rng(11)
    x, w, dy = _rand_pair(rng, g, 20)
    st, pd = g.stride_h, g.pad_h
    tx, tw, tdy = (torch.from_numpy(v.astype(np.float64)) for v in (x, w, dy))
    y_ref = torch.nn.functional.conv2d(tx, tw, stride=st, padding=pd).numpy()
    dx_ref = torch.nn.grad.conv2d_input(tx.shape, tw, tdy, stride=st, padding=pd).numpy()
    dw_ref = torch.nn.grad.conv2d_weight(tx, tw.shape, tdy, stride=st, padding=pd).numpy()
    big = 10 ** 7
    y, _, _ = orc.conv(g, orc.FWD, x, w, 0, big)
    dx, _, _ = orc.conv(g, orc.BWD_DATA, dy, w, 0, big)
    dw, _, _ = orc.conv(g, orc.BWD_WT, x, dy, 0, big)
    assert np.array_equal(y.astype(np.float64), y_ref)
    assert np.array_equal(dx.astype(np.float64), dx_ref)
    assert np.array_equal(dw.astype(np.float64), dw_ref)


@pytest.mark.parametrize("L", [1, 2, 5, 9, 64])
def test_multi_chunk_exact_values_equal_torch_scaled(orc, L):
    """With small integers every FP32 partial sum is exact, so chunking changes
    nothing and the output is the exact convolution times 2^(Ea+Eb)."""
    g = orc.geom(2, 6, 8, 7, 5, 3, 3, 1, 1)
    rng = np.random.default_rng(12)
    x, w, dy = _rand_pair(rng, g, 30)
    tx, tw, tdy = (torch.from_numpy(v.astype(np.float64)) for v in (x, w, dy))
    e = -9
    y, _, _ = orc.conv(g, orc.FWD, x, w, e, L)
    ref = torch.nn.functional.conv2d(tx, tw, padding=1).numpy() * 2.0 ** e
    assert np.array_equal(y.astype(np.float64), ref)
    for G in (1, 2, 7, 0):
        dw, _, _ = orc.conv(g, orc.BWD_WT, x, dy, e, L, G)
        ref = torch.nn.grad.conv2d_weight(tx, tw.shape, tdy, padding=1).numpy() * 2.0 ** e
        assert np.array_equal(dw.astype(np.float64), ref)


# ------------------------------------------------------ adjoint identity --
@pytest.mark.parametrize("shape", SHAPES)
def test_adjoint_identity(orc, shape):
    """<fwd(x,w), dy> = <x, bwd_data(dy,w)> = <w, bwd_wt(x,dy)>, exact in int64."""
    g = orc.geom(*shape)
    rng = np.random.default_rng(13)
    x, w, dy = _rand_pair(rng, g, 40)
    big = 10 ** 7
    y, _, _ = orc.conv(g, orc.FWD, x, w, 0, big)
    dx, _, _ = orc.conv(g, orc.BWD_DATA, dy, w, 0, big)
    dw, _, _ = orc.conv(g, orc.BWD_WT, x, dy, 0, big)
    a = int((y.astype(np.int64) * dy.astype(np.int64)).sum())
    b = int((x.astype(np.int64) * dx.astype(np.int64)).sum())
    c = int((w.astype(np.int64) * dw.astype(np.int64)).sum())
    assert a == b == c


# ------------------------------------------------ overflow figures --------
def test_sec43_three_products_overflow(orc):
    """Sec. 4.3: an INT16 product is a 30-bit value and a chain of three such
    products can overflow INT32; two cannot.  32767^2 * 2 = 2,147,352,578 fits;
    * 3 = 3,221,028,867 wraps to -1,073,938,429."""
    g = orc.geom(1, 3, 1, 1, 1, 1, 1)
    x = np.full((1, 3, 1, 1), 32767, np.int16)
    w = np.full((1, 3, 1, 1), 32767, np.int16)
    y, parts, ov = orc.conv(g, orc.FWD, x, w, 0, 3, want_partials=True)
    assert ov == 1 and int(parts[0, 0]) == -1073938429 and float(y[0, 0, 0, 0]) == float(np.float32(-1073938429))
    y, parts, ov = orc.conv(g, orc.FWD, x, w, 0, 2, want_partials=True)
    assert ov == 0 and [int(v) for v in parts[:, 0]] == [2147352578, 1073676289]
    assert float(y[0, 0, 0, 0]) == float(np.float32(np.float32(2147352578) + np.float32(1073676289)))


def test_dfp15_wraps_only_at_eight(orc):
    """DFP15 operands are at most 2^14 in magnitude, products at most 2^28:
    7 of them fit INT32, 8 reach 2^31 and wrap to -2^31."""
    g = orc.geom(1, 8, 1, 1, 1, 1, 1)
    x = np.full((1, 8, 1, 1), 16384, np.int16)
    w = np.full((1, 8, 1, 1), 16384, np.int16)
    _, parts, ov = orc.conv(g, orc.FWD, x, w, 0, 8, want_partials=True)
    assert ov == 1 and int(parts[0, 0]) == -2 ** 31
    _, parts, ov = orc.conv(g, orc.FWD, x, w, 0, 7, want_partials=True)
    assert ov == 0 and [int(v) for v in parts[:, 0]] == [7 * 2 ** 28, 2 ** 28]


# ------------------------------------------- canonical reduction order ----
def test_one_hot_products_land_in_their_chunk(orc):
    """A single nonzero product at tap (r, s), channel c lands in chunk
    t // L with t = (r*S + s)*C + c (fwd), (r*S + s)*K + k (bwd-data),
    (n*P + p)*Q + q (bwd-wt)."""
    n, C, H, W, K, R, S = 2, 5, 6, 6, 3, 3, 3
    g = orc.geom(n, C, H, W, K, R, S, 1, 1)
    L = 4
    rng = np.random.default_rng(14)
    for _ in range(25):
        c, r, s, k = (int(rng.integers(0, v)) for v in (C, R, S, K))
        nn, p, q = int(rng.integers(0, n)), int(rng.integers(1, H - 1)), int(rng.integers(1, W - 1))
        ih, iw = p - 1 + r, q - 1 + s
        x = np.zeros((n, C, H, W), np.int16)
        x[nn, c, ih, iw] = 3
        w = np.zeros((K, C, R, S), np.int16)
        w[k, c, r, s] = 5
        dy = np.zeros((n, K, H, W), np.int16)
        dy[nn, k, p, q] = 7
        # fwd output (nn, k, p, q)
        _, parts, _ = orc.conv(g, orc.FWD, x, w, 0, L, want_partials=True)
        o = ((nn * K + k) * H + p) * W + q
        j = ((r * S + s) * C + c) // L
        assert parts[j, o] == 15 and np.count_nonzero(parts) == 1
        # bwd-data output (nn, c, ih, iw)
        _, parts, _ = orc.conv(g, orc.BWD_DATA, dy, w, 0, L, want_partials=True)
        o = ((nn * C + c) * H + ih) * W + iw
        j = ((r * S + s) * K + k) // L
        assert parts[j, o] == 35 and np.count_nonzero(parts) == 1
        # bwd-wt output (k, c, r, s)
        _, parts, _ = orc.conv(g, orc.BWD_WT, x, dy, 0, L, want_partials=True)
        o = ((k * C + c) * R + r) * S + s
        j = ((nn * H + p) * W + q) // L
        assert parts[j, o] == 21 and np.count_nonzero(parts) == 1


# -------------------------------------------------- FP32 chain ------------
def test_fp32_chain_error_bound_and_float32_replay(orc):
    """|y - exact*2^E| <= ((J-1) u sum|F_j| + u sum|P_j|) 2^E (recursive
    summation plus conversion rounding), and the sequential float32 replay
    of the partials in numpy gives the same bits."""
    g = orc.geom(2, 64, 7, 7, 8, 3, 3, 1, 1)
    rng = np.random.default_rng(15)
    x, w, dy = _rand_pair(rng, g, 2 ** 14)
    e = -26
    exact = brute_fwd(x, w, 1, 1).reshape(-1)
    u = 2.0 ** -24
    for L in (8, 16, 64):
        y, parts, ov = orc.conv(g, orc.FWD, x, w, e, L, want_partials=True)
        if ov:
            continue
        F = parts.astype(np.float32)
        J = parts.shape[0]
        bound = ((J - 1) * u * np.abs(F.astype(np.float64)).sum(0) + u * np.abs(parts.astype(np.float64)).sum(0))
        err = np.abs(y.reshape(-1).astype(np.float64) - exact.astype(np.float64) * 2.0 ** e)
        assert np.all(err <= bound * 2.0 ** e + 1e-300)
        acc = F[0].copy()
        for j in range(1, J):
            acc = (acc + F[j]).astype(np.float32)
        assert np.array_equal(np.ldexp(acc.astype(np.float64), e).astype(np.float32), y.reshape(-1))


def test_bwd_wt_segments(orc):
    """G = 1 and G = J are both the plain sequential sum over chunks; any G
    obeys the summation error bound."""
    g = orc.geom(4, 3, 9, 9, 4, 3, 3, 1, 1)
    rng = np.random.default_rng(16)
    x, w, dy = _rand_pair(rng, g, 2 ** 14)
    L = 5
    J = orc.num_chunks(g, orc.BWD_WT, L)
    a, parts, ov = orc.conv(g, orc.BWD_WT, x, dy, 0, L, 1, want_partials=True)
    b, _, _ = orc.conv(g, orc.BWD_WT, x, dy, 0, L, J)
    assert np.array_equal(a, b)
    exact = wrap32(parts.astype(np.int64)).astype(np.float64).sum(0)
    for G in (2, 3, 17):
        c, _, _ = orc.conv(g, orc.BWD_WT, x, dy, 0, L, G)
        bound = J * 2.0 ** -24 * np.abs(parts.astype(np.float64)).sum(0) * 2
        assert np.all(np.abs(c.reshape(-1) - exact) <= bound)


def _segment_fold_float32(parts, G, e):
    """Sec. 4.3 reading C8 replayed in numpy float32 from the chunk partials:
    each segment of G consecutive chunks summed in chunk order (the last
    segment possibly shorter), then the segment sums in segment order, then
    one rounding of the sum times 2^e."""
    F = parts.astype(np.float32)
    J = F.shape[0]
    seg_sums = []
    for g0 in range(0, J, G):
        u = F[g0].copy()
        for j in range(g0 + 1, min(J, g0 + G)):
            u = (u + F[j]).astype(np.float32)
        seg_sums.append(u)
    s = seg_sums[0].copy()
    for u in seg_sums[1:]:
        s = (s + u).astype(np.float32)
    return np.ldexp(s.astype(np.float64), e).astype(np.float32)


@pytest.mark.parametrize("G", [2, 3, 16, 17])
def test_bwd_wt_segment_fold_float32_replay(orc, G):
    """The oracle's two-level backward-weights sum equals an independent
    float32 replay of its own partials bit for bit, for segment sizes whose
    last segment is only partly filled (J = 65 chunks: 1, 2, 1 and 14 chunks
    in the last segment) and with large-magnitude operands so that the
    float32 additions round."""
    g = orc.geom(4, 3, 9, 9, 4, 3, 3, 1, 1)
    rng = np.random.default_rng(161)
    x, _, dy = _rand_pair(rng, g, 2 ** 14)
    L, e = 5, -23
    J = orc.num_chunks(g, orc.BWD_WT, L)
    assert J == 65 and J % G != 0
    y, parts, _ = orc.conv(g, orc.BWD_WT, x, dy, e, L, G, want_partials=True)
    ref = _segment_fold_float32(parts, G, e)
    assert np.array_equal(y.reshape(-1).view(np.uint32), ref.view(np.uint32))
    # the replay is sensitive to the segment boundaries: a neighbouring G differs somewhere
    other = _segment_fold_float32(parts, G + 1, e)
    assert not np.array_equal(other.view(np.uint32), ref.view(np.uint32))


# ---------------------------------------------------- linearity mod 2^32 --
def test_partials_linear_mod_2_32(orc):
    g = orc.geom(1, 16, 5, 5, 3, 3, 3, 1, 1)
    rng = np.random.default_rng(17)
    x1 = rng.integers(-2 ** 13, 2 ** 13, (1, 16, 5, 5)).astype(np.int16)
    x2 = rng.integers(-2 ** 13, 2 ** 13, (1, 16, 5, 5)).astype(np.int16)
    w = rng.integers(-2 ** 14, 2 ** 14, (3, 16, 3, 3)).astype(np.int16)
    L = 32
    _, p1, _ = orc.conv(g, orc.FWD, x1, w, 0, L, want_partials=True)
    _, p2, _ = orc.conv(g, orc.FWD, x2, w, 0, L, want_partials=True)
    _, p3, _ = orc.conv(g, orc.FWD, (x1.astype(np.int32) + x2).astype(np.int16), w, 0, L, want_partials=True)
    assert np.array_equal(wrap32(p1.astype(np.int64) + p2), p3.astype(np.int64))


# ----------------------------------------------- sampled == full ----------
def test_conv_at_matches_full(orc):
    g = orc.geom(2, 5, 7, 6, 4, 3, 3, 2, 1)
    rng = np.random.default_rng(18)
    x, w, dy = _rand_pair(rng, g, 2 ** 14)
    for d, a, b in ((orc.FWD, x, w), (orc.BWD_DATA, dy, w), (orc.BWD_WT, x, dy)):
        full, parts, _ = orc.conv(g, d, a, b, -20, 6, 3, want_partials=True)
        idx = rng.choice(full.size, size=min(40, full.size), replace=False)
        vals, pp, _ = orc.conv_at(g, d, a, b, -20, 6, idx, 3, want_partials=True)
        assert np.array_equal(vals, full.reshape(-1)[idx])
        assert np.array_equal(pp, parts[:, idx].T)


def test_scale_extremes(orc):
    """The scale 2^(Ea+Eb) is applied once with a single rounding: results may
    be subnormal (rounded once) or overflow to inf."""
    g = orc.geom(1, 1, 1, 1, 1, 1, 1)
    x = np.array(3, np.int16).reshape(1, 1, 1, 1)
    w = np.array(1, np.int16).reshape(1, 1, 1, 1)
    y, _, _ = orc.conv(g, orc.FWD, x, w, -150, 4)  # 3 * 2^-150 = 1.5 * 2^-149 -> ties to even: 2^-148
    assert float(y.reshape(-1)[0]) == 2.0 ** -148
    y, _, _ = orc.conv(g, orc.FWD, x, w, 127, 4)
    assert np.isinf(y).all() and orc.output_flags(y) == orc.FLAG_OUTPUT_INF

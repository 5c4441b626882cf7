"""Pins of the oracle's GEMM (the forward convolution's chunked contract,
Alg. 2 and Sec. 4.3, applied to a matrix product) against references outside
it: numpy's int64 matrix product (a library routine) for exact results and
for every chunk partial modulo 2^32, a worked example of the FP32 chunk-order
fold, and the oracle's 1x1 forward convolution (a separately pinned route)."""
import numpy as np
import pytest

import oracle

TRANS = [(False, False), (False, True), (True, False), (True, True)]


def stored(op_a, op_b, ta, tb):
    """The arrays as the GEMM reads them for logical operands opA [m,k], opB [k,n]."""
    a = np.ascontiguousarray(op_a.T if ta else op_a)
    b = np.ascontiguousarray(op_b.T if tb else op_b)
    return a, b


def wrap32(v):
    return ((v.astype(np.int64) + 2 ** 31) % 2 ** 32 - 2 ** 31).astype(np.int64)


@pytest.mark.parametrize("ta,tb", TRANS)
def test_single_chunk_small_values_equal_numpy(ta, tb):
    rng = np.random.default_rng(1)
    m, n, k = 13, 17, 200
    op_a = rng.integers(-100, 101, (m, k)).astype(np.int16)
    op_b = rng.integers(-100, 101, (k, n)).astype(np.int16)
    a, b = stored(op_a, op_b, ta, tb)
    e = -7
    d, parts, ov = oracle.gemm(a, b, e, 256, ta, tb, want_partials=True)
    exact = op_a.astype(np.int64) @ op_b.astype(np.int64)  # |.| < 2^24: exact in FP32
    assert ov == 0
    assert np.array_equal(parts[0].reshape(m, n), exact)
    assert np.array_equal(d, (exact * 2.0 ** e).astype(np.float32))


@pytest.mark.parametrize("ta,tb", TRANS)
@pytest.mark.parametrize("L", [1, 7, 32, 64, 1003])
def test_partials_are_wrapped_chunk_products(ta, tb, L):
    rng = np.random.default_rng([2, L, ta, tb])
    m, n, k = 9, 11, 1000
    op_a = rng.integers(-32767, 32768, (m, k)).astype(np.int16)
    op_b = rng.integers(-32767, 32768, (k, n)).astype(np.int16)
    a, b = stored(op_a, op_b, ta, tb)
    d, parts, ov = oracle.gemm(a, b, 0, L, ta, tb, want_partials=True)
    J = (k + L - 1) // L
    assert parts.shape == (J, m * n)
    wrapped = 0
    for c in range(J):
        sl = slice(c * L, min(k, (c + 1) * L))
        ex = op_a[:, sl].astype(np.int64) @ op_b[sl, :].astype(np.int64)
        assert np.array_equal(parts[c].reshape(m, n), wrap32(ex)), c
        wrapped += int(np.count_nonzero(wrap32(ex) != ex))
    assert ov == wrapped
    if L >= 64:
        assert ov > 0  # 64 full-range products exceed 2^31


def test_fold_is_fp32_in_chunk_order():
    # chunk partials 2^25, 1, 1, 1, 1 (L = 1): adding in chunk order in FP32
    # keeps 2^25 at every step (the spacing there is 4); the exact sum 2^25 + 4
    # is representable, so any other order or a wider accumulator differs
    a = np.array([[8192, 1, 1, 1, 1]], dtype=np.int16)
    b = np.array([[4096], [1], [1], [1], [1]], dtype=np.int16)
    d, parts, _ = oracle.gemm(a, b, 0, 1, want_partials=True)
    assert list(parts[:, 0]) == [2 ** 25, 1, 1, 1, 1]
    assert d[0, 0] == np.float32(2 ** 25)
    d2, _, _ = oracle.gemm(a[:, ::-1].copy(), b[::-1].copy(), 0, 1)
    assert d2[0, 0] == np.float32(2 ** 25 + 4)
    d3, _, _ = oracle.gemm(a, b, -25, 5)  # one chunk: the exact sum, then the scale
    assert d3[0, 0] == np.float32(1 + 4 * 2.0 ** -25)


@pytest.mark.parametrize("L", [5, 16, 64])
def test_equals_one_by_one_forward_convolution(L):
    # D = W X is the 1x1 forward convolution of x [1, k, 1, n] with w [m, k, 1, 1]
    rng = np.random.default_rng(L)
    m, n, k = 24, 37, 150
    w = rng.integers(-16384, 16385, (m, k)).astype(np.int16)
    x = rng.integers(-16384, 16385, (k, n)).astype(np.int16)
    g = oracle.geom(1, k, 1, n, m, 1, 1)
    y, py, _ = oracle.conv(g, 0, x.reshape(1, k, 1, n), w.reshape(m, k, 1, 1), -20, L, want_partials=True)
    d, pd, _ = oracle.gemm(w, x, -20, L, want_partials=True)
    assert np.array_equal(pd, py)
    assert np.array_equal(d.reshape(-1), y.reshape(-1))


def test_scale_applied_once_with_gradual_underflow():
    a = np.array([[3, 5]], dtype=np.int16)
    b = np.array([[7], [11]], dtype=np.int16)
    d, _, _ = oracle.gemm(a, b, -140, 1)  # 21 + 55 = 76, times 2^-140: a subnormal
    assert d[0, 0] == np.float32(np.ldexp(76.0, -140))
    d, _, _ = oracle.gemm(a, b, 122, 1)  # 76 * 2^122 > FP32 max
    assert np.isinf(d[0, 0])

"""Pins of the oracle's Blocked-DFP (Sec. 3: several exponents per tensor,
each shared by a small block of integers) against references outside it: the
single-exponent quantiser when one block spans the tensor, the quantiser
applied block by block, Eq. 2's placement of every block maximum, the
unblocked GEMM when all exponents agree, an exact closed form with differing
block exponents, and a worked example of the per-chunk scaled fold."""
import numpy as np
import pytest

import oracle

MODES = ["nearest", "stochastic", "biased", "down"]


@pytest.mark.parametrize("rounding", MODES)
@pytest.mark.parametrize("bits", [15, 16])
def test_one_block_is_the_single_exponent_quantiser(rounding, bits):
    rng = np.random.default_rng(bits)
    f = (rng.standard_normal((1, 5003)) * 7).astype(np.float32)
    q, e, fl = oracle.quantize_blocked(f, 8192, bits, oracle.ROUNDING[rounding], 99, oracle.ROLE_W)
    rq, re, rfl = oracle.quantize(f.reshape(-1), bits, oracle.ROUNDING[rounding], 99, oracle.ROLE_W)
    assert np.array_equal(q.reshape(-1), rq)
    assert e.shape == (1, 1) and int(e[0, 0]) == re
    assert fl == rfl


@pytest.mark.parametrize("B", [1, 3, 32, 64, 100])
def test_blocks_are_quantised_independently(B):
    # nearest rounding draws nothing, so each block equals the quantiser on that block alone
    rng = np.random.default_rng(B)
    rows, cols = 7, 333
    scale = np.exp2(rng.integers(-20, 20, (rows, cols))).astype(np.float32)  # wide dynamic range
    f = (rng.standard_normal((rows, cols)) * scale).astype(np.float32)
    q, e, _ = oracle.quantize_blocked(f, B, 15, oracle.ROUND_NEAREST)
    nb = (cols + B - 1) // B
    assert e.shape == (nb, rows)
    for r in range(rows):
        for b in range(nb):
            blk = f[r, b * B:(b + 1) * B]
            rq, re, _ = oracle.quantize(blk, 15, oracle.ROUND_NEAREST)
            assert np.array_equal(q[r, b * B:(b + 1) * B], rq)
            assert int(e[b, r]) == re


@pytest.mark.parametrize("rounding", MODES)
def test_every_block_max_sits_at_bit_p_minus_2(rounding):
    rng = np.random.default_rng(3)
    f = (rng.standard_normal((16, 256)) * np.exp2(rng.integers(-30, 30, (16, 1)))).astype(np.float32)
    q, e, _ = oracle.quantize_blocked(f, 64, 15, oracle.ROUNDING[rounding], 5)
    for r in range(16):
        for b in range(4):
            blk = q[r, b * 64:(b + 1) * 64].astype(np.int64)
            mx = np.abs(blk).max()
            assert 2 ** 13 <= mx <= 2 ** 14  # Eq. 2 with P = 15: max lands at bit 13 (rounding may reach 2^14)
            # dequantised block within one step of the FP32 values
            x = f[r, b * 64:(b + 1) * 64].astype(np.float64) * 2.0 ** -int(e[b, r])
            assert np.all(np.abs(blk - x) < 1.0 + 1e-12)


def test_zero_and_nonfinite_blocks():
    f = np.zeros((2, 8), dtype=np.float32)
    f[1, 4] = np.inf
    f[1, 5] = 3.0
    q, e, fl = oracle.quantize_blocked(f, 4, 15, oracle.ROUND_NEAREST)
    assert fl == oracle.FLAG_NONFINITE  # not ZERO_TENSOR: one block is non-finite
    assert not q.any() and not e.any()
    q, e, fl = oracle.quantize_blocked(np.zeros((3, 5), np.float32), 2, 15, oracle.ROUND_NEAREST)
    assert fl == oracle.FLAG_ZERO_TENSOR
    g = np.zeros((1, 8), dtype=np.float32)
    g[0, 6] = 1.0
    q, e, fl = oracle.quantize_blocked(g, 4, 15, oracle.ROUND_NEAREST)
    assert fl == 0 and list(e[:, 0]) == [0, -13] and q[0, 6] == 2 ** 13


@pytest.mark.parametrize("L,Bk", [(32, 32), (32, 128), (64, 64), (16, 64)])
def test_equal_exponents_match_the_unblocked_gemm(L, Bk):
    rng = np.random.default_rng(L + Bk)
    m, n, k = 9, 13, 300
    a = rng.integers(-16384, 16385, (m, k)).astype(np.int16)
    b = rng.integers(-16384, 16385, (n, k)).astype(np.int16)
    nb = (k + Bk - 1) // Bk
    ea = np.full((nb, m), -12, np.int8)
    eb = np.full((nb, n), -9, np.int8)
    d, p, _ = oracle.gemm_blocked(a, ea, b, eb, Bk, L, want_partials=True)
    rd, rp, _ = oracle.gemm(a, b, -21, L, trans_b=True, want_partials=True)
    assert np.array_equal(p, rp)
    assert np.array_equal(d, rd)  # scaling each chunk or the sum by 2^-21 agree away from underflow


def test_closed_form_with_block_exponents():
    rng = np.random.default_rng(8)
    m, n, k, Bk = 5, 6, 96, 32
    a = rng.integers(-10, 11, (m, k)).astype(np.int16)
    b = rng.integers(-10, 11, (n, k)).astype(np.int16)
    ea = rng.integers(-2, 3, (3, m)).astype(np.int8)
    eb = rng.integers(-2, 3, (3, n)).astype(np.int8)
    d, _, _ = oracle.gemm_blocked(a, ea, b, eb, Bk, 32)
    # |block sum| <= 3200 < 2^12 and scales 2^-4 .. 2^4: every term and partial
    # sum is a multiple of 2^-4 below 2^18, so FP32 holds all of them exactly
    exact = np.zeros((m, n))
    for blk in range(3):
        s = a[:, blk * 32:(blk + 1) * 32].astype(np.int64) @ b[:, blk * 32:(blk + 1) * 32].T.astype(np.int64)
        exact += s * np.exp2(ea[blk][:, None].astype(np.int64) + eb[blk][None, :].astype(np.int64))
    assert np.array_equal(d, exact.astype(np.float32))
    assert np.array_equal(d.astype(np.float64), exact)


def test_fold_scales_each_chunk_then_adds_in_order():
    # five chunks of one product each (L = Bk = 1): block 0 scaled by 2^25, the
    # rest by 2^0; in chunk order the FP32 sum stays at 2^25, while the exact
    # sum 2^25 + 4 is representable
    a = np.ones((1, 5), np.int16)
    b = np.ones((1, 5), np.int16)
    ea = np.array([[25], [0], [0], [0], [0]], np.int8)
    eb = np.zeros((5, 1), np.int8)
    d, _, _ = oracle.gemm_blocked(a, ea, b, eb, 1, 1)
    assert d[0, 0] == np.float32(2 ** 25)
    d2, _, _ = oracle.gemm_blocked(a, ea[::-1].copy(), b, eb, 1, 1)
    assert d2[0, 0] == np.float32(2 ** 25 + 4)

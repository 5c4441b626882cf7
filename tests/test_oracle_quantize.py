"""Pins for the oracle's quantiser (Sec. 3.1 Eq. 1-3, rounding modes of Sec. 1).

Nothing here re-types the oracle's own procedure: the oracle rounds through an
exact fraction word F = floor(frac(x) * 2^32); these tests compare it with
library routines that implement the textbook modes directly (np.rint,
np.floor), hand-derived worked examples, and invariants that any correct
quantiser must satisfy.
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
HELPERS = os.path.join(os.path.dirname(__file__), "helpers")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


# ---------------------------------------------------------------- Philox ---
def test_philox_known_answers(orc):
    for row in _rows("philox4x32_10_kat.txt"):
        v = [int(t, 16) for t in row]
        out = orc.philox4x32_10(v[0:4], v[4:6])
        assert [int(o) for o in out] == v[6:10]


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not available")
def test_philox_stream_matches_rocrand(orc, tmp_path):
    exe = tmp_path / "rr"
    subprocess.check_call(["hipcc", "-x", "hip", "--offload-arch=gfx950", "-O1", "-w",
                           os.path.join(HELPERS, "rocrand_philox.cpp"), "-o", str(exe)])
    rng = np.random.default_rng(7)
    queries = [(int(rng.integers(0, 2**64, dtype=np.uint64)), int(rng.integers(0, 5)),
                int(rng.integers(0, 2**40))) for _ in range(300)]
    queries += [(0, 0, i) for i in range(16)] + [(1, 4, 2**32 * 4 + 3), (2**64 - 1, 2, 2**34 + 1)]
    text = "".join("%d %d %d\n" % q for q in queries)
    out = subprocess.run([str(exe)], input=text, capture_output=True, text=True, check=True).stdout.split()
    assert len(out) == len(queries)
    for (seed, role, idx), ref in zip(queries, out):
        assert orc.rng_word(seed, role, idx) == int(ref), (seed, role, idx)


def test_philox_words_uniform(orc):
    # chi-square over 16 bins of the top 4 bits: 8192 words, df = 15
    words = np.array([orc.rng_word(12345, 0, i) for i in range(8192)], dtype=np.uint64)
    counts = np.bincount((words >> 28).astype(np.int64), minlength=16)
    exp = len(words) / 16
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 40.0  # p ~ 5e-4 for df=15


# ------------------------------------------------------ worked examples ---
def test_worked_example(orc):
    rows = list(_rows("quantize_worked_example.txt"))
    f = np.array([float(r[0]) for r in rows], dtype=np.float32)
    modes = {"nearest": 2, "biased": 3, "down": 4}
    for mode, col in modes.items():
        i, es, flags = orc.quantize(f, 15, orc.ROUNDING[mode])
        assert es == -13 and flags == 0
        assert [int(v) for v in i] == [int(r[col]) for r in rows], mode
    # stochastic: P(up) = F / 2^32 ; over many seeds the empirical rate matches
    S = 4000
    ups = np.zeros(len(f))
    for seed in range(S):
        i, es, _ = orc.quantize(f, 15, orc.ROUND_STOCHASTIC, seed)
        fl = np.floor(f.astype(np.float64) * 2.0 ** 13)
        ups += (i - fl)
    p = np.array([int(r[5]) for r in rows], dtype=np.float64) / 2.0 ** 32
    tol = 5 * np.sqrt(p * (1 - p) / S) + 1e-9
    assert np.all(np.abs(ups / S - p) <= tol)


def test_rounding_ties(orc):
    rows = list(_rows("rounding_ties.txt"))
    f = np.array([float(r[0]) for r in rows], dtype=np.float32)
    for mode, col in (("nearest", 2), ("biased", 3), ("down", 4)):
        i, es, flags = orc.quantize(f, 15, orc.ROUNDING[mode])
        assert es == -1
        assert [int(v) for v in i] == [int(r[col]) for r in rows], mode


# --------------------------------------------- library special cases ---
def _adversarial(rng, n, emax):
    """float32 values with |f| <= 2^emax: normals, subnormals, exact ties,
    values one ulp around ties, small integers, zeros."""
    parts = [
        rng.standard_normal(n).astype(np.float32) * np.float32(2.0 ** (emax - 3)),
        (rng.integers(-2**20, 2**20, n) * 2.0 ** (emax - 21)).astype(np.float32),
        ((rng.integers(-2**13, 2**13, n) + 0.5) * 2.0 ** (emax - 13)).astype(np.float32),
        np.array([0.0, -0.0], dtype=np.float32),
    ]
    ties = parts[2]
    parts.append(np.nextafter(ties, np.float32(np.inf)))
    parts.append(np.nextafter(ties, np.float32(-np.inf)))
    sub = rng.integers(1, 2**23, n).astype(np.uint32).view(np.float32)  # subnormals
    parts.append(sub * np.where(rng.random(n) < 0.5, -1, 1).astype(np.float32))
    f = np.concatenate(parts).astype(np.float32)
    f = np.clip(f, -np.float32(2.0 ** emax), np.float32(2.0 ** emax))
    return np.concatenate([np.array([np.float32(2.0 ** emax) * np.float32(1.5)], dtype=np.float32), f])


@pytest.mark.parametrize("emax", [-140, -20, 0, 7, 60, 126])
def test_modes_equal_library_rounding(orc, emax):
    rng = np.random.default_rng(1000 + emax)
    f = _adversarial(rng, 20000, emax)
    for bits in (15, 16):
        ref_i, es, flags = orc.quantize(f, bits, orc.ROUND_NEAREST)
        x = f.astype(np.float64) * 2.0 ** (-es)  # exact in float64
        lim = 32767 if bits == 16 else 2**20
        assert np.array_equal(ref_i, np.clip(np.rint(x), -lim, lim).astype(np.int16))
        i, es2, _ = orc.quantize(f, bits, orc.ROUND_BIASED)
        assert es2 == es and np.array_equal(i, np.clip(np.floor(x + 0.5), -lim, lim).astype(np.int16))
        i, es2, _ = orc.quantize(f, bits, orc.ROUND_DOWN)
        assert es2 == es and np.array_equal(i, np.clip(np.floor(x), -lim, lim).astype(np.int16))
        # stochastic always lands on floor(x) or floor(x)+1
        i, es2, _ = orc.quantize(f, bits, orc.ROUND_STOCHASTIC, seed=99)
        d = i.astype(np.float64) - np.floor(x)
        assert es2 == es and np.all((d == 0) | (d == 1) | (np.abs(i) == 32767))


def test_bitpattern_sweep(orc):
    """Strided sweep of all FP32 bit patterns below a fixed max (a CPU-sized
    stand-in for the exhaustive sweep), against np.rint / np.floor(x + 0.5)."""
    step = 65537
    bits_ = np.arange(0, 0x7f800000, step, dtype=np.uint64).astype(np.uint32)
    mags = bits_.view(np.float32)
    for top in (np.float32(1.0), np.float32(3.0e38), np.float32(2.0 ** -126)):
        f = mags[mags <= top]
        f = np.concatenate([[top], f, -f]).astype(np.float32)
        i, es, _ = orc.quantize(f, 15, orc.ROUND_NEAREST)
        x = f.astype(np.float64) * 2.0 ** (-es)
        assert np.array_equal(i, np.rint(x).astype(np.int16))
        i, _, _ = orc.quantize(f, 15, orc.ROUND_BIASED)
        assert np.array_equal(i, np.floor(x + 0.5).astype(np.int16))


# ------------------------------------------------------------ invariants ---
@pytest.mark.parametrize("bits", [15, 16])
def test_max_lands_at_bit_p_minus_2(orc, bits):
    rng = np.random.default_rng(bits)
    for scale in (1e-30, 1e-3, 1.0, 37.0, 1e30):
        f = (rng.standard_normal(5000) * scale).astype(np.float32)
        i, es, flags = orc.quantize(f, bits, orc.ROUND_NEAREST)
        m = int(np.abs(i.astype(np.int64)).max())
        assert 2 ** (bits - 2) <= m <= 2 ** (bits - 1)
        # the shared exponent reproduces the max within the rounding step
        assert abs(float(np.abs(f).max()) - m * 2.0 ** es) <= 2.0 ** (es - 1)


def test_nearest_error_bound(orc):
    rng = np.random.default_rng(3)
    for dist in range(4):
        f = rng.standard_normal(20000).astype(np.float32)
        if dist == 1:
            f = np.maximum(f, 0)
        if dist == 2:
            f = f * np.float32(1e-3)
        if dist == 3:
            f = np.exp(rng.standard_normal(20000) * 8).astype(np.float32)
        i, es, _ = orc.quantize(f, 15, orc.ROUND_NEAREST)
        err = np.abs(f.astype(np.float64) - i.astype(np.float64) * 2.0 ** es)
        assert err.max() <= 2.0 ** (es - 1)


def test_scale_invariance(orc):
    rng = np.random.default_rng(4)
    f = rng.standard_normal(4096).astype(np.float32)
    for mode in range(4):
        i0, e0, _ = orc.quantize(f, 15, mode, seed=5)
        for k in (-40, -3, 1, 17, 60):
            i1, e1, _ = orc.quantize((f * np.float32(2.0 ** k)).astype(np.float32), 15, mode, seed=5)
            assert e1 == e0 + k and np.array_equal(i0, i1)


def test_nearest_odd_symmetry(orc):
    rng = np.random.default_rng(5)
    f = _adversarial(rng, 3000, 3)
    i0, e0, _ = orc.quantize(f, 15, orc.ROUND_NEAREST)
    i1, e1, _ = orc.quantize(-f, 15, orc.ROUND_NEAREST)
    assert e0 == e1 and np.array_equal(i1, -i0)


def test_special_tensors(orc):
    z = np.zeros(100, dtype=np.float32)
    i, es, flags = orc.quantize(z, 15)
    assert es == 0 and not i.any() and flags == orc.FLAG_ZERO_TENSOR
    bad = np.ones(10, dtype=np.float32)
    for v in (np.inf, -np.inf, np.nan):
        bad[3] = v
        i, es, flags = orc.quantize(bad, 15)
        assert flags == orc.FLAG_NONFINITE and es == 0 and not i.any()
    # max 2^-116: Efmax - 13 = -129 is below the 8-bit range and clamps to -128
    tiny = np.array([2.0 ** -116, -(2.0 ** -117), 2.0 ** -149], dtype=np.float32)
    i, es, flags = orc.quantize(tiny, 15)
    assert es == -128 and flags == orc.FLAG_EXP_CLAMPED
    assert list(i) == [2 ** 12, -(2 ** 11), 0]


def test_p16_saturation(orc):
    # x_max = 32767.75 rounds to 32768 and must clamp to 32767 (only P = 16)
    top = np.float32(32767.75 * 2.0 ** -14)
    f = np.array([top, -top, 0.5], dtype=np.float32)
    i, es, flags = orc.quantize(f, 16, orc.ROUND_NEAREST)
    assert es == -14 and list(i[:2]) == [32767, -32767] and flags & orc.FLAG_SATURATED
    i, es, flags = orc.quantize(f, 15, orc.ROUND_NEAREST)
    assert es == -13 and list(i[:2]) == [16384, -16384] and flags == 0


def test_stochastic_unbiased(orc):
    rng = np.random.default_rng(6)
    f = np.concatenate([[np.float32(1.0)], rng.uniform(-1, 1, 63)]).astype(np.float32)
    S = 4096
    acc = np.zeros(f.size)
    for seed in range(S):
        i, es, _ = orc.quantize(f, 15, orc.ROUND_STOCHASTIC, seed=seed, role=2)
        acc += i
    x = f.astype(np.float64) * 2.0 ** 13
    p = x - np.floor(x)
    tol = 5 * np.sqrt(p * (1 - p) / S) + 2.0 ** -32
    assert np.all(np.abs(acc / S - x) <= tol)


def test_stochastic_streams_differ_by_role_and_seed(orc):
    f = np.linspace(-1, 1, 1001).astype(np.float32)
    a, _, _ = orc.quantize(f, 15, orc.ROUND_STOCHASTIC, seed=1, role=0)
    b, _, _ = orc.quantize(f, 15, orc.ROUND_STOCHASTIC, seed=1, role=1)
    c, _, _ = orc.quantize(f, 15, orc.ROUND_STOCHASTIC, seed=2, role=0)
    d, _, _ = orc.quantize(f, 15, orc.ROUND_STOCHASTIC, seed=1, role=0)
    assert not np.array_equal(a, b) and not np.array_equal(a, c) and np.array_equal(a, d)


# ------------------------------------------------ Eq. 6 down-conversion ---
def test_eq6_worked_example(orc):
    # i = 2^20 + 5 has 11 leading zeros in 32 bits.  Read literally, Eq. 6 gives
    # Rs = 32 - (16 + 11) = 5 and 2^15 + 0 = 32768, which does not fit INT16;
    # placing the max at bit P-2 (as Eq. 2 does) gives Rs = 6 -> 16384 at P = 16.
    src = np.array([2 ** 20 + 5, -3, 1000], dtype=np.int32)
    i, e, flags = orc.downconvert_i32(src, 0, bits=16, rounding=orc.ROUND_DOWN)
    assert e == 6 and int(i[0]) == 16384
    i, e, flags = orc.downconvert_i32(src, 10, bits=15, rounding=orc.ROUND_NEAREST)
    assert e == 17 and int(i[0]) == 8192 and int(i[2]) == 8


def test_eq6_equals_float_quantisation(orc):
    """Eq. 6 on <I, E> equals Eq. 1-3 applied to the exact values I * 2^E."""
    rng = np.random.default_rng(8)
    for scale_bits in (3, 14, 20, 30):
        src = rng.integers(-2 ** scale_bits, 2 ** scale_bits, 5000).astype(np.int32)
        for e_in in (-30, 0, 5):
            vals = src.astype(np.float64) * 2.0 ** e_in
            if scale_bits > 24:  # keep the float32 image exact: drop low bits first
                src = (src >> (scale_bits - 24)) << (scale_bits - 24)
                vals = src.astype(np.float64) * 2.0 ** e_in
            f = vals.astype(np.float32)
            assert np.array_equal(f.astype(np.float64), vals)
            for mode in range(4):
                a, ea, _ = orc.downconvert_i32(src, e_in, 15, mode, seed=3, role=3)
                b, eb, _ = orc.quantize(f, 15, mode, seed=3, role=3)
                assert ea == eb and np.array_equal(a, b)

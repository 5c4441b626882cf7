"""GPU parity of dfp_quantize / dfp_downconvert against the CPU oracle:
INT16 tensors, exponents and flags bit-exact, for every rounding mode, both
bit widths, ragged sizes and the special tensors."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV, note, to_dev
from paper_1802_00930_amd import dfp

pytestmark = pytest.mark.gpu


def role_desc(n, bits, rounding, seed, role):
    """A descriptor whose tensor of the given role holds exactly n elements."""
    if role == dfp.ROLE_W:
        return dfp.make_desc(1, 1, 1, 1, n, 1, 1, bits=bits, rounding=rounding, seed=seed)
    return dfp.make_desc(1, 1, 1, n, 1, 1, 1, bits=bits, rounding=rounding, seed=seed)


def gpu_quant(f, bits, rounding, seed, role):
    n = f.size
    d = role_desc(n, bits, rounding, seed, role)
    t = to_dev(f.astype(np.float32))
    out = torch.empty(t.shape, dtype=torch.int16, device=DEV)
    sc = dfp.new_scale(DEV)
    if role in (dfp.ROLE_Y, dfp.ROLE_DX):
        dfp.dfp_downconvert(d, role, t, out, sc, amax_ready=False)
    else:
        dfp.dfp_quantize(d, role, t, out, sc)
    torch.cuda.synchronize()
    return out.cpu().numpy().reshape(-1), dfp.read_scale(sc)


def check(f, bits, rounding, seed=0, role=0):
    f = np.ascontiguousarray(f, dtype=np.float32).reshape(-1)
    gi, sc = gpu_quant(f, bits, rounding, seed, role)
    oi, oe, ofl = oracle.quantize(f, bits, rounding, seed, role)
    assert sc["exp"] == oe, (sc, oe)
    assert sc["flags"] == ofl, (sc, ofl)
    bad = np.nonzero(gi != oi.reshape(-1))[0]
    assert bad.size == 0, "mismatch at %s: gpu %s oracle %s f %s" % (bad[:5], gi[bad[:5]], oi.reshape(-1)[bad[:5]],
                                                                     f[bad[:5]])
    # amax_bits: the max of |f| bit patterns
    if not ofl & oracle.FLAG_NONFINITE:
        assert sc["amax_bits"] == int((f.view(np.uint32) & 0x7fffffff).max())


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 8, 63, 1000, 4097, 65535, 65536, 65537, (1 << 20) + 3])
@pytest.mark.parametrize("rounding", [0, 1, 2, 3])
def test_sizes_and_modes(n, rounding):
    rng = np.random.default_rng(n * 7 + rounding)
    f = rng.standard_normal(n).astype(np.float32)
    note("quantize n=%d rounding=%d" % (n, rounding))
    for bits in (15, 16):
        check(f, bits, rounding, seed=n, role=dfp.ROLE_X)


@pytest.mark.parametrize("role", [0, 1, 2, 3, 4])
def test_roles_and_seeds(role):
    rng = np.random.default_rng(100 + role)
    f = np.maximum(rng.standard_normal(50001), 0).astype(np.float32) * np.float32(1e-3)
    for seed in (0, 1, 2 ** 40 + 17, 2 ** 64 - 1):
        note("quantize role=%d seed=%d" % (role, seed))
        check(f, 15, oracle.ROUND_STOCHASTIC, seed=seed, role=role)


@pytest.mark.parametrize("scale", [1e-38, 1e-20, 1e-3, 1.0, 3e4, 1e30, 3e38])
def test_magnitudes(scale):
    rng = np.random.default_rng(int(np.log10(scale) + 100))
    f = (rng.standard_normal(20000) * scale).astype(np.float32)
    f = f[np.isfinite(f)]
    note("quantize scale=%g" % scale)
    for rounding in range(4):
        for bits in (15, 16):
            check(f, bits, rounding, seed=3)


def test_ties_and_neighbours():
    rng = np.random.default_rng(5)
    ties = ((rng.integers(-2 ** 13, 2 ** 13, 30000) + 0.5) * 2.0 ** -3).astype(np.float32)
    f = np.concatenate([[np.float32(1024.0)], ties, np.nextafter(ties, np.float32(9e9)),
                        np.nextafter(ties, np.float32(-9e9))]).astype(np.float32)
    for rounding in range(4):
        for bits in (15, 16):
            check(f, bits, rounding, seed=11)


def test_special_tensors():
    check(np.zeros(1000, np.float32), 15, 0)
    for v in (np.inf, -np.inf, np.nan):
        f = np.ones(999, np.float32)
        f[500] = v
        check(f, 15, 0)
        check(f, 16, 1)
    check(np.array([2.0 ** -116, -(2.0 ** -117), 2.0 ** -149, 0.0], np.float32), 15, 0)  # exponent clamp
    top = np.float32(32767.75 * 2.0 ** -14)
    check(np.array([top, -top, 0.5, 1e-3], np.float32), 16, 0)  # P=16 saturation
    check(np.array([top, -top, 0.5, 1e-3], np.float32), 16, 2)
    sub = (np.arange(1, 5000, dtype=np.uint32) * 977).view(np.float32)  # subnormals only
    check(sub, 15, 0)
    check(-sub, 16, 1, seed=4)


@pytest.mark.parametrize("top_bits", [0x3f800000, 0x7f7fffff, 0x00800000, 0x00000fff, 0x4b000000])
def test_bitpattern_sweep(top_bits):
    """Every 61st FP32 bit pattern up to a chosen max (both signs), so each
    E_s sees patterns from every binade below its max."""
    pats = np.arange(0, top_bits + 1, 61, dtype=np.uint64).astype(np.uint32)
    mags = pats.view(np.float32)
    top = np.array([top_bits], np.uint32).view(np.float32)
    f = np.concatenate([top, mags, -mags]).astype(np.float32)
    note("quantize sweep top=0x%08x n=%d" % (top_bits, f.size))
    for rounding in (0, 1, 2):
        check(f, 15, rounding, seed=7)
    check(f, 16, 0)

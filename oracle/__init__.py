"""CPU oracle for DFP INT16 convolution -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg
may import this package.  The product library (``paper_1802_00930_amd``) never
imports, links or calls it, and it shares no code with the HIP path.

Thin ctypes wrapper around ``dfp_oracle.c`` (plain C, float64/int64 exact
arithmetic, one output at a time).  Each function below states the passage of
Das et al. (ICLR 2018) it follows; the C file lists the readings taken where the
paper is silent.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dfp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ROUND_NEAREST, ROUND_STOCHASTIC, ROUND_BIASED, ROUND_DOWN = 0, 1, 2, 3
ROUNDING = {"nearest": 0, "stochastic": 1, "biased": 2, "down": 3}
ROLE_X, ROLE_W, ROLE_DY, ROLE_Y, ROLE_DX = 0, 1, 2, 3, 4
FWD, BWD_DATA, BWD_WT = 0, 1, 2

FLAG_NONFINITE = 1
FLAG_EXP_CLAMPED = 2
FLAG_SATURATED = 4
FLAG_ZERO_TENSOR = 8
FLAG_OUTPUT_INF = 16


def build(force: bool = False) -> str:
    """Compile dfp_oracle.c into liboracle.so (gcc -O2 -fopenmp, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-fno-fast-math", "-ffp-contract=off", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class Geom(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        L = ctypes.CDLL(build())
        P = ctypes.c_void_p
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_philox4x32_10.restype = None
        L.orc_rng_word.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64]
        L.orc_rng_word.restype = ctypes.c_uint32
        L.orc_quantize.argtypes = [P, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_uint64,
                                   ctypes.c_uint32, P, P]
        L.orc_quantize.restype = ctypes.c_uint32
        L.orc_downconvert_i32.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_uint64, ctypes.c_uint32, P, P]
        L.orc_downconvert_i32.restype = ctypes.c_uint32
        L.orc_conv.argtypes = [ctypes.POINTER(Geom), ctypes.c_int, P, P, ctypes.c_int32, ctypes.c_int32,
                               ctypes.c_int32, P, P]
        L.orc_conv.restype = ctypes.c_int64
        L.orc_conv_at.argtypes = [ctypes.POINTER(Geom), ctypes.c_int, P, P, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_int32, P, ctypes.c_int64, P, P]
        L.orc_conv_at.restype = ctypes.c_int64
        L.orc_num_chunks.argtypes = [ctypes.POINTER(Geom), ctypes.c_int, ctypes.c_int32]
        L.orc_num_chunks.restype = ctypes.c_int64
        L.orc_output_len.argtypes = [ctypes.POINTER(Geom), ctypes.c_int]
        L.orc_output_len.restype = ctypes.c_int64
        L.orc_default_seg_chunks.argtypes = [ctypes.c_int32]
        L.orc_default_seg_chunks.restype = ctypes.c_int32
        L.orc_output_flags.argtypes = [P, ctypes.c_int64]
        L.orc_output_flags.restype = ctypes.c_uint32
        L.orc_gemm.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int, P, P,
                               ctypes.c_int32, ctypes.c_int32, P, P]
        L.orc_gemm.restype = ctypes.c_int64
        L.orc_quantize_blocked.argtypes = [P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_uint64, ctypes.c_uint32, P, P]
        L.orc_quantize_blocked.restype = ctypes.c_uint32
        L.orc_gemm_blocked.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, P, P, P, P, ctypes.c_int64,
                                       ctypes.c_int32, P, P]
        L.orc_gemm_blocked.restype = ctypes.c_int64
        I64, I32, F = ctypes.c_int64, ctypes.c_int32, ctypes.c_float
        L.orc_bn_relu_fwd.argtypes = [P, I32, I64, I64, I64, P, P, P, F, ctypes.c_int, ctypes.c_int, ctypes.c_uint64,
                                      P, P, P, P, P, P]
        L.orc_bn_relu_fwd.restype = ctypes.c_uint32
        L.orc_bn_relu_bwd.argtypes = [P, I32, P, I32, I64, I64, I64, P, P, P, P, P, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_uint64, P, P, P, P, P, P, P]
        L.orc_bn_relu_bwd.restype = ctypes.c_uint32
        L.orc_sgd_quantize.argtypes = [I64, P, P, P, F, F, F, ctypes.c_int, ctypes.c_int, ctypes.c_uint64, P, P]
        L.orc_sgd_quantize.restype = ctypes.c_uint32
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def geom(n, c, h, w, k, r, s, stride=1, pad=0, stride_w=None, pad_w=None) -> Geom:
    return Geom(n, c, h, w, k, r, s, stride, stride if stride_w is None else stride_w,
                pad, pad if pad_w is None else pad_w)


def out_hw(g: Geom):
    return ((g.h + 2 * g.pad_h - g.r) // g.stride_h + 1, (g.w + 2 * g.pad_w - g.s) // g.stride_w + 1)


# --------------------------------------------------------------------------
# Philox4x32-10 (Salmon et al., SC'11): the counter-based generator that draws
# the uniforms for stochastic rounding (the paper names the rounding mode,
# Sec. 1, but no generator).
# --------------------------------------------------------------------------
def philox4x32_10(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def rng_word(seed: int, role: int, idx: int) -> int:
    return int(lib().orc_rng_word(seed, role, idx))


# --------------------------------------------------------------------------
# Quantisation FP32 -> DFP-P: shared exponent from the max magnitude (Eq. 1-2),
# integers such that f ~ i * 2^Es (Eq. 3), rounded with the requested mode
# (Sec. 1).  Also used for the down-conversion of a conv output (Sec. 4.1).
# --------------------------------------------------------------------------
def quantize(f: np.ndarray, bits: int = 15, rounding: int = ROUND_NEAREST, seed: int = 0,
             role: int = ROLE_X):
    f = np.ascontiguousarray(f, dtype=np.float32)
    out = np.empty(f.shape, dtype=np.int16)
    es = np.zeros(1, dtype=np.int32)
    flags = lib().orc_quantize(_ptr(f), f.size, bits, rounding, seed, role, _ptr(out), _ptr(es))
    return out, int(es[0]), int(flags)


def downconvert_i32(i32: np.ndarray, e_in: int, bits: int = 15, rounding: int = ROUND_NEAREST,
                    seed: int = 0, role: int = ROLE_Y):
    """Eq. 6 (integer DFP-32 -> DFP-P), with the shift count placing the max at
    bit P-2 as Eq. 2 does."""
    src = np.ascontiguousarray(i32, dtype=np.int32)
    out = np.empty(src.shape, dtype=np.int16)
    es = np.zeros(1, dtype=np.int32)
    flags = lib().orc_downconvert_i32(_ptr(src), src.size, e_in, bits, rounding, seed, role,
                                      _ptr(out), _ptr(es))
    return out, int(es[0]), int(flags)


# --------------------------------------------------------------------------
# Convolutions (Alg. 2 and Sec. 4.3): INT32 partials over chunks of L products,
# FP32 sum in chunk order, one scale 2^(Ea+Eb) (Eq. 4).
# --------------------------------------------------------------------------
def num_chunks(g: Geom, direction: int, L: int) -> int:
    return int(lib().orc_num_chunks(ctypes.byref(g), direction, L))


def default_seg_chunks(L: int) -> int:
    return int(lib().orc_default_seg_chunks(L))


def _out_shape(g: Geom, direction: int):
    P, Q = out_hw(g)
    if direction == FWD:
        return (g.n, g.k, P, Q)
    if direction == BWD_DATA:
        return (g.n, g.c, g.h, g.w)
    return (g.k, g.c, g.r, g.s)


def conv(g: Geom, direction: int, a: np.ndarray, b: np.ndarray, e: int, L: int, G: int = 0,
         want_partials: bool = False):
    """Returns (out float32, partials int32 [J, outputs] or None, wrapped-partial count).

    fwd: a = x, b = w; bwd-data: a = dy, b = w; bwd-wt: a = x, b = dy; e = Ea + Eb."""
    a = np.ascontiguousarray(a, dtype=np.int16)
    b = np.ascontiguousarray(b, dtype=np.int16)
    shape = _out_shape(g, direction)
    out = np.empty(shape, dtype=np.float32)
    parts = None
    if want_partials:
        J = num_chunks(g, direction, L)
        parts = np.empty((J, out.size), dtype=np.int32)
    ov = lib().orc_conv(ctypes.byref(g), direction, _ptr(a), _ptr(b), e, L, G, _ptr(out),
                        _ptr(parts) if parts is not None else None)
    return out, parts, int(ov)


def conv_at(g: Geom, direction: int, a: np.ndarray, b: np.ndarray, e: int, L: int, idx, G: int = 0,
            want_partials: bool = False):
    """The same as :func:`conv` at the flat output indices ``idx`` only.
    Returns (values float32 [len], partials int32 [len, J] or None, wrapped count)."""
    a = np.ascontiguousarray(a, dtype=np.int16)
    b = np.ascontiguousarray(b, dtype=np.int16)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.float32)
    parts = None
    if want_partials:
        J = num_chunks(g, direction, L)
        parts = np.empty((idx.size, J), dtype=np.int32)
    ov = lib().orc_conv_at(ctypes.byref(g), direction, _ptr(a), _ptr(b), e, L, G, _ptr(idx), idx.size,
                           _ptr(out), _ptr(parts) if parts is not None else None)
    return out, parts, int(ov)


def output_flags(y: np.ndarray) -> int:
    y = np.ascontiguousarray(y, dtype=np.float32)
    return int(lib().orc_output_flags(_ptr(y), y.size))


# --------------------------------------------------------------------------
# GEMM with the forward convolution's chunked contract (Alg. 2, Sec. 4.3; the
# paper's kernels serve "convolutions and GEMM", Sec. 4).
# --------------------------------------------------------------------------
def gemm(a: np.ndarray, b: np.ndarray, e: int, L: int, trans_a: bool = False, trans_b: bool = False,
         want_partials: bool = False):
    """D = opA @ opB with INT32 partials over chunks of L reduction indices,
    FP32 sum in chunk order, scale 2^e.  a is stored [m, k] (or [k, m] with
    trans_a), b [k, n] (or [n, k] with trans_b).  Returns (D float32 [m, n],
    partials int32 [J, m*n] or None, wrapped-partial count)."""
    a = np.ascontiguousarray(a, dtype=np.int16)
    b = np.ascontiguousarray(b, dtype=np.int16)
    m, k = (a.shape[1], a.shape[0]) if trans_a else a.shape
    kb, n = (b.shape[1], b.shape[0]) if trans_b else b.shape
    assert k == kb, (a.shape, b.shape, trans_a, trans_b)
    out = np.empty((m, n), dtype=np.float32)
    parts = np.empty(((k + L - 1) // L, m * n), dtype=np.int32) if want_partials else None
    ov = lib().orc_gemm(m, n, k, int(trans_a), int(trans_b), _ptr(a), _ptr(b), e, L, _ptr(out),
                        _ptr(parts) if parts is not None else None)
    return out, parts, int(ov)


# --------------------------------------------------------------------------
# Blocked-DFP (Sec. 3): one exponent per block of B consecutive elements of a
# row; a GEMM over such operands scales each chunk by its block's exponents
# before the FP32 fold (Alg. 2).
# --------------------------------------------------------------------------
def quantize_blocked(f: np.ndarray, B: int, bits: int = 15, rounding: int = ROUND_NEAREST, seed: int = 0,
                     role: int = ROLE_X):
    """f [rows, cols] FP32 -> (int16 [rows, cols], int8 exponents [nb, rows], flags)."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    rows, cols = f.shape
    nb = (cols + B - 1) // B
    out = np.empty((rows, cols), dtype=np.int16)
    exps = np.empty((nb, rows), dtype=np.int8)
    flags = lib().orc_quantize_blocked(_ptr(f), rows, cols, B, bits, rounding, seed, role, _ptr(out), _ptr(exps))
    return out, exps, int(flags)


def gemm_blocked(a: np.ndarray, ea: np.ndarray, b: np.ndarray, eb: np.ndarray, Bk: int, L: int,
                 want_partials: bool = False):
    """a [m, k], b [n, k] INT16 (t contiguous), ea [nb, m], eb [nb, n] int8;
    D [m, n] = fold over chunks of 2^(ea + eb) * fl32(P_c).  Bk % L == 0."""
    assert Bk % L == 0
    a = np.ascontiguousarray(a, dtype=np.int16)
    b = np.ascontiguousarray(b, dtype=np.int16)
    ea = np.ascontiguousarray(ea, dtype=np.int8)
    eb = np.ascontiguousarray(eb, dtype=np.int8)
    m, k = a.shape
    n = b.shape[0]
    assert b.shape[1] == k and ea.shape == ((k + Bk - 1) // Bk, m) and eb.shape == ((k + Bk - 1) // Bk, n)
    out = np.empty((m, n), dtype=np.float32)
    parts = np.empty(((k + L - 1) // L, m * n), dtype=np.int32) if want_partials else None
    ov = lib().orc_gemm_blocked(m, n, k, _ptr(a), _ptr(ea), _ptr(b), _ptr(eb), Bk, L, _ptr(out),
                                _ptr(parts) if parts is not None else None)
    return out, parts, int(ov)


# --------------------------------------------------------------------------
# The steps either side of the convolutions in one training step (Sec. 4.1,
# Fig. 2): batch normalisation on up-converted DFP16 tensors with ReLU and an
# optional residual add, the quantisers Q_a / Q_e of its outputs, and FP32 SGD
# on master weights followed by Q_w.  Channel sums are exact integers.
# --------------------------------------------------------------------------
def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def bn_relu_fwd(y: np.ndarray, ey: int, gamma, beta, res=None, eps: float = 1e-5, bits: int = 15,
                rounding: int = ROUND_NEAREST, seed: int = 0):
    """y int16 [N, C, H, W] with exponent ey.  Returns dict: z (FP32), zq, ez,
    flags, mean, inv_std (FP32 [C]), sums (int64 [C, 2]: S1, S2)."""
    y = np.ascontiguousarray(y, dtype=np.int16)
    N, C = y.shape[:2]
    HW = y[0, 0].size
    g, b, r = _f32(gamma), _f32(beta), _f32(res)
    z = np.empty(y.shape, np.float32)
    zq = np.empty(y.shape, np.int16)
    ez = np.zeros(1, np.int32)
    mean = np.empty(C, np.float32)
    inv = np.empty(C, np.float32)
    sums = np.empty((C, 2), np.int64)
    fl = lib().orc_bn_relu_fwd(_ptr(y), ey, N, C, HW, _ptr(g), _ptr(b), _ptr(r) if r is not None else None, eps,
                               bits, rounding, seed, _ptr(z), _ptr(zq), _ptr(ez), _ptr(mean), _ptr(inv), _ptr(sums))
    return dict(z=z, zq=zq, ez=int(ez[0]), flags=int(fl), mean=mean, inv_std=inv, sums=sums)


def bn_relu_bwd(dz: np.ndarray, edz: int, y: np.ndarray, ey: int, gamma, beta, mean, inv_std, res=None,
                bits: int = 15, rounding: int = ROUND_NEAREST, seed: int = 0):
    """Returns dict: dy (FP32), dyq, edy, flags, dgamma, dbeta, dres (FP32 or
    None), sums (int64 [C, 2]: D, P)."""
    dz = np.ascontiguousarray(dz, dtype=np.int16)
    y = np.ascontiguousarray(y, dtype=np.int16)
    N, C = y.shape[:2]
    HW = y[0, 0].size
    g, b, r, m, s = _f32(gamma), _f32(beta), _f32(res), _f32(mean), _f32(inv_std)
    dy = np.empty(y.shape, np.float32)
    dyq = np.empty(y.shape, np.int16)
    edy = np.zeros(1, np.int32)
    dg = np.empty(C, np.float32)
    db = np.empty(C, np.float32)
    dres = np.empty(y.shape, np.float32) if r is not None else None
    sums = np.empty((C, 2), np.int64)
    fl = lib().orc_bn_relu_bwd(_ptr(dz), edz, _ptr(y), ey, N, C, HW, _ptr(g), _ptr(b),
                               _ptr(r) if r is not None else None, _ptr(m), _ptr(s), bits, rounding, seed, _ptr(dy),
                               _ptr(dyq), _ptr(edy), _ptr(dg), _ptr(db), _ptr(dres) if dres is not None else None,
                               _ptr(sums))
    return dict(dy=dy, dyq=dyq, edy=int(edy[0]), flags=int(fl), dgamma=dg, dbeta=db, dres=dres, sums=sums)


def sgd_quantize(w, v, dw, lr: float, mu: float, wd: float, bits: int = 15, rounding: int = ROUND_NEAREST,
                 seed: int = 0):
    """One FP32 SGD step (returns new copies of w and v) and Q_w of the new w."""
    w = np.array(w, dtype=np.float32, copy=True).reshape(-1)
    v = np.array(v, dtype=np.float32, copy=True).reshape(-1)
    dw = _f32(dw).reshape(-1)
    wq = np.empty(w.size, np.int16)
    ew = np.zeros(1, np.int32)
    fl = lib().orc_sgd_quantize(w.size, _ptr(w), _ptr(v), _ptr(dw), lr, mu, wd, bits, rounding, seed, _ptr(wq),
                                _ptr(ew))
    return dict(w=w, v=v, wq=wq, ew=int(ew[0]), flags=int(fl))

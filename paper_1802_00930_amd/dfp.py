"""Python binding of libdfp (argument marshalling only).

Every function here has the name of a C entry point in ``include/dfp.h`` and
does nothing but check tensor dtypes/devices and pass raw device pointers,
sizes and the current HIP stream to it.  All computation happens in the HIP
kernels of ``libdfp.so``; there is no fallback.  PyTorch supplies device
memory and streams only.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdfp.so")

OK, ERR_NULL, ERR_SHAPE, ERR_PARAM, ERR_ALIGN, ERR_WORKSPACE, ERR_HIP, ERR_SCRATCH_LIMIT = range(8)
NOALLOC_SCRATCH_BYTES = 64 << 20
ROUND_NEAREST, ROUND_STOCHASTIC, ROUND_BIASED, ROUND_DOWN = range(4)
ROUNDING = {"nearest": 0, "stochastic": 1, "biased": 2, "down": 3}
ROLE_X, ROLE_W, ROLE_DY, ROLE_Y, ROLE_DX = range(5)
FWD, BWD_DATA, BWD_WT = range(3)
PATH_AUTO, PATH_MFMA, PATH_VALU = range(3)
FLAG_NONFINITE, FLAG_EXP_CLAMPED, FLAG_SATURATED, FLAG_ZERO_TENSOR, FLAG_OUTPUT_INF = 1, 2, 4, 8, 16


class DfpError(RuntimeError):
    def __init__(self, func, status):
        super().__init__("%s failed: %s (%d)" % (func, status_str(status), status))
        self.status = status


class Desc(ctypes.Structure):
    """Mirror of ``dfp_desc``."""
    _fields_ = [(name, ctypes.c_int32) for name in
                ("n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
                 "chunk_len", "seg_chunks", "bits", "rounding", "path")] + [("seed", ctypes.c_uint64)]


class BnDesc(ctypes.Structure):
    """Mirror of ``dfp_bn_desc``."""
    _fields_ = [(name, ctypes.c_int32) for name in ("n", "c", "hw", "bits", "rounding")] + \
        [("eps", ctypes.c_float), ("seed", ctypes.c_uint64)]


class GemmDesc(ctypes.Structure):
    """Mirror of ``dfp_gemm_desc``."""
    _fields_ = [(name, ctypes.c_int32) for name in
                ("m", "n", "k", "trans_a", "trans_b", "chunk_len", "bits", "path")]


_lib = None


def lib():
    """Load libdfp.so; raise if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libdfp.so is not built at %s; run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        DP = ctypes.POINTER(Desc)
        GP = ctypes.POINTER(GemmDesc)
        BP = ctypes.POINTER(BnDesc)
        F = ctypes.c_float
        sigs = {
            "dfp_quantize": ([DP, I32, P, P, P, P], I32),
            "dfp_conv_fwd": ([DP, P, P, P, P, P, P, P, SZ, P, P], I32),
            "dfp_conv_bwd_data": ([DP, P, P, P, P, P, P, P, SZ, P, P], I32),
            "dfp_conv_bwd_weights": ([DP, P, P, P, P, P, P, SZ, P, P], I32),
            "dfp_conv_bwd_weights_noalloc": ([DP, P, P, P, P, P, P], I32),
            "dfp_downconvert": ([DP, I32, P, P, P, I32, P], I32),
            "dfp_conv_fwd_i32": ([DP, P, P, P, P, P, P, P, SZ, P], I32),
            "dfp_conv_bwd_data_i32": ([DP, P, P, P, P, P, P, P, SZ, P], I32),
            "dfp_downconvert_i32": ([DP, I32, P, P, P, P, I32, P], I32),
            "dfp_workspace_bytes": ([DP, I32], SZ),
            "dfp_gemm": ([GP, P, P, P, P, P, P, P, SZ, P, P], I32),
            "dfp_gemm_workspace_bytes": ([GP], SZ),
            "dfp_gemm_num_chunks": ([GP], I64),
            "dfp_quantize_tensor": ([I64, I32, I32, ctypes.c_uint64, I32, P, P, P, P], I32),
            "dfp_quantize_blocked": ([I64, I64, I64, I32, I32, ctypes.c_uint64, I32, P, P, P, P, P], I32),
            "dfp_gemm_blocked": ([GP, I32, P, P, P, P, P, P, P, SZ, P, P], I32),
            "dfp_gemm_blocked_workspace_bytes": ([GP, I32], SZ),
            "dfp_downconvert_tensor": ([I64, I32, I32, ctypes.c_uint64, I32, P, P, P, I32, P], I32),
            "dfp_num_chunks": ([DP, I32], I64),
            "dfp_output_dims": ([DP, ctypes.POINTER(I32), ctypes.POINTER(I32)], I32),
            "dfp_bn_workspace_bytes": ([BP], SZ),
            "dfp_bn_relu_fwd": ([BP, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
            "dfp_bn_relu_bwd": ([BP, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
            "dfp_sgd_quantize": ([I64, F, F, F, I32, I32, ctypes.c_uint64, P, P, P, P, P, P], I32),
            "dfp_status_str": ([I32], ctypes.c_char_p),
            "dfp_profile_start": ([I32], I32),
            "dfp_profile_stop": ([P, P, I32], I32),
            "dfp_kernel_name": ([I32], ctypes.c_char_p),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().dfp_status_str(status).decode()


def make_desc(n, c, h, w, k, r, s, stride=1, pad=0, chunk_len=64, seg_chunks=0, bits=15,
              rounding="nearest", path=PATH_AUTO, seed=0, stride_w=None, pad_w=None) -> Desc:
    rnd = ROUNDING[rounding] if isinstance(rounding, str) else int(rounding)
    return Desc(n, c, h, w, k, r, s, stride, stride if stride_w is None else stride_w, pad,
                pad if pad_w is None else pad_w, chunk_len, seg_chunks, bits, rnd, path, seed)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, dtype, what):
    if t is None:
        return
    if not t.is_cuda or t.dtype != dtype or not t.is_contiguous():
        raise TypeError("%s must be a contiguous %s CUDA tensor" % (what, dtype))


def _check(func, status):
    if status != OK:
        raise DfpError(func, status)


def new_scale(device="cuda") -> torch.Tensor:
    """A zeroed dfp_scale (16 bytes: amax_bits, exp, flags, reserved) as int32[4]."""
    return torch.zeros(4, dtype=torch.int32, device=device)


def read_scale(scale: torch.Tensor) -> dict:
    v = scale.cpu().tolist()
    return {"amax_bits": v[0] & 0xffffffff, "exp": v[1], "flags": v[2] & 0xffffffff}


def output_dims(d: Desc):
    p, q = ctypes.c_int32(), ctypes.c_int32()
    _check("dfp_output_dims", lib().dfp_output_dims(ctypes.byref(d), ctypes.byref(p), ctypes.byref(q)))
    return p.value, q.value


def num_chunks(d: Desc, direction: int) -> int:
    return int(lib().dfp_num_chunks(ctypes.byref(d), direction))


def workspace_bytes(d: Desc, direction: int) -> int:
    return int(lib().dfp_workspace_bytes(ctypes.byref(d), direction))


def dfp_quantize(d: Desc, role: int, src, dst, scale, stream=None):
    _need(src, torch.float32, "src"); _need(dst, torch.int16, "dst"); _need(scale, torch.int32, "scale")
    _check("dfp_quantize", lib().dfp_quantize(ctypes.byref(d), role, _ptr(src), _ptr(dst), _ptr(scale),
                                              _stream(stream)))


def dfp_downconvert(d: Desc, role: int, src, dst, scale, amax_ready: bool = False, stream=None):
    _need(src, torch.float32, "src"); _need(dst, torch.int16, "dst"); _need(scale, torch.int32, "scale")
    _check("dfp_downconvert", lib().dfp_downconvert(ctypes.byref(d), role, _ptr(src), _ptr(dst), _ptr(scale),
                                                    int(bool(amax_ready)), _stream(stream)))


def _ws(workspace):
    if workspace is None:
        return None, 0
    return _ptr(workspace), workspace.numel() * workspace.element_size()


def dfp_conv_fwd(d: Desc, x, sx, w, sw, y, sy=None, workspace=None, partials=None, stream=None):
    for t, dt, nm in ((x, torch.int16, "x"), (w, torch.int16, "w"), (y, torch.float32, "y"),
                      (sx, torch.int32, "sx"), (sw, torch.int32, "sw"), (sy, torch.int32, "sy"),
                      (partials, torch.int32, "partials")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_conv_fwd", lib().dfp_conv_fwd(ctypes.byref(d), _ptr(x), _ptr(sx), _ptr(w), _ptr(sw), _ptr(y),
                                              _ptr(sy), wp, wn, _ptr(partials), _stream(stream)))


def dfp_conv_bwd_data(d: Desc, dy, sdy, w, sw, dx, sdx=None, workspace=None, partials=None, stream=None):
    for t, dt, nm in ((dy, torch.int16, "dy"), (w, torch.int16, "w"), (dx, torch.float32, "dx"),
                      (sdy, torch.int32, "sdy"), (sw, torch.int32, "sw"), (sdx, torch.int32, "sdx"),
                      (partials, torch.int32, "partials")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_conv_bwd_data", lib().dfp_conv_bwd_data(ctypes.byref(d), _ptr(dy), _ptr(sdy), _ptr(w), _ptr(sw),
                                                        _ptr(dx), _ptr(sdx), wp, wn, _ptr(partials),
                                                        _stream(stream)))


def dfp_conv_bwd_weights(d: Desc, x, sx, dy, sdy, dw, workspace=None, partials=None, stream=None):
    for t, dt, nm in ((x, torch.int16, "x"), (dy, torch.int16, "dy"), (dw, torch.float32, "dw"),
                      (sx, torch.int32, "sx"), (sdy, torch.int32, "sdy"), (partials, torch.int32, "partials")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_conv_bwd_weights", lib().dfp_conv_bwd_weights(ctypes.byref(d), _ptr(x), _ptr(sx), _ptr(dy),
                                                              _ptr(sdy), _ptr(dw), wp, wn, _ptr(partials),
                                                              _stream(stream)))


def dfp_conv_bwd_weights_noalloc(d: Desc, x, sx, dy, sdy, dw, stream=None):
    for t, dt, nm in ((x, torch.int16, "x"), (dy, torch.int16, "dy"), (dw, torch.float32, "dw"),
                      (sx, torch.int32, "sx"), (sdy, torch.int32, "sdy")):
        _need(t, dt, nm)
    _check("dfp_conv_bwd_weights_noalloc",
           lib().dfp_conv_bwd_weights_noalloc(ctypes.byref(d), _ptr(x), _ptr(sx), _ptr(dy), _ptr(sdy), _ptr(dw),
                                              _stream(stream)))


def dfp_conv_fwd_i32(d: Desc, x, sx, w, sw, y, sy, workspace=None, stream=None):
    for t, dt, nm in ((x, torch.int16, "x"), (w, torch.int16, "w"), (y, torch.int32, "y"),
                      (sx, torch.int32, "sx"), (sw, torch.int32, "sw"), (sy, torch.int32, "sy")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_conv_fwd_i32", lib().dfp_conv_fwd_i32(ctypes.byref(d), _ptr(x), _ptr(sx), _ptr(w), _ptr(sw),
                                                      _ptr(y), _ptr(sy), wp, wn, _stream(stream)))


def dfp_conv_bwd_data_i32(d: Desc, dy, sdy, w, sw, dx, sdx, workspace=None, stream=None):
    for t, dt, nm in ((dy, torch.int16, "dy"), (w, torch.int16, "w"), (dx, torch.int32, "dx"),
                      (sdy, torch.int32, "sdy"), (sw, torch.int32, "sw"), (sdx, torch.int32, "sdx")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_conv_bwd_data_i32", lib().dfp_conv_bwd_data_i32(ctypes.byref(d), _ptr(dy), _ptr(sdy), _ptr(w),
                                                                _ptr(sw), _ptr(dx), _ptr(sdx), wp, wn,
                                                                _stream(stream)))


def dfp_downconvert_i32(d: Desc, role: int, src, sin, dst, sout, amax_ready: bool = False, stream=None):
    for t, dt, nm in ((src, torch.int32, "src"), (dst, torch.int16, "dst"), (sin, torch.int32, "sin"),
                      (sout, torch.int32, "sout")):
        _need(t, dt, nm)
    _check("dfp_downconvert_i32", lib().dfp_downconvert_i32(ctypes.byref(d), role, _ptr(src), _ptr(sin), _ptr(dst),
                                                            _ptr(sout), int(bool(amax_ready)), _stream(stream)))


def make_gemm_desc(m, n, k, trans_a=False, trans_b=False, chunk_len=64, bits=15, path=PATH_AUTO) -> GemmDesc:
    return GemmDesc(m, n, k, int(bool(trans_a)), int(bool(trans_b)), chunk_len, bits, path)


def gemm_workspace_bytes(d: GemmDesc) -> int:
    return int(lib().dfp_gemm_workspace_bytes(ctypes.byref(d)))


def gemm_num_chunks(d: GemmDesc) -> int:
    return int(lib().dfp_gemm_num_chunks(ctypes.byref(d)))


def alloc_gemm_workspace(d: GemmDesc, device="cuda"):
    n = gemm_workspace_bytes(d)
    if n == 0:
        return None
    return torch.empty((n + 255) // 256 * 256, dtype=torch.uint8, device=device)


def dfp_gemm(d: GemmDesc, a, sa, b, sb, out, sd=None, workspace=None, partials=None, stream=None):
    for t, dt, nm in ((a, torch.int16, "a"), (b, torch.int16, "b"), (out, torch.float32, "out"),
                      (sa, torch.int32, "sa"), (sb, torch.int32, "sb"), (sd, torch.int32, "sd"),
                      (partials, torch.int32, "partials")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_gemm", lib().dfp_gemm(ctypes.byref(d), _ptr(a), _ptr(sa), _ptr(b), _ptr(sb), _ptr(out), _ptr(sd),
                                      wp, wn, _ptr(partials), _stream(stream)))


def dfp_quantize_tensor(bits, rounding, seed, role, src, dst, scale, stream=None):
    _need(src, torch.float32, "src"); _need(dst, torch.int16, "dst"); _need(scale, torch.int32, "scale")
    rnd = ROUNDING[rounding] if isinstance(rounding, str) else int(rounding)
    _check("dfp_quantize_tensor", lib().dfp_quantize_tensor(src.numel(), bits, rnd, seed, role, _ptr(src),
                                                            _ptr(dst), _ptr(scale), _stream(stream)))


def dfp_downconvert_tensor(bits, rounding, seed, role, src, dst, scale, amax_ready=False, stream=None):
    _need(src, torch.float32, "src"); _need(dst, torch.int16, "dst"); _need(scale, torch.int32, "scale")
    rnd = ROUNDING[rounding] if isinstance(rounding, str) else int(rounding)
    _check("dfp_downconvert_tensor", lib().dfp_downconvert_tensor(src.numel(), bits, rnd, seed, role, _ptr(src),
                                                                  _ptr(dst), _ptr(scale), int(bool(amax_ready)),
                                                                  _stream(stream)))


def dfp_quantize_blocked(block, bits, rounding, seed, role, src, dst, exps, scale, stream=None):
    """src: FP32 [rows, cols]; dst INT16 like src; exps int8 [ceil(cols/block), rows]."""
    _need(src, torch.float32, "src"); _need(dst, torch.int16, "dst"); _need(exps, torch.int8, "exps")
    _need(scale, torch.int32, "scale")
    rows, cols = src.shape
    rnd = ROUNDING[rounding] if isinstance(rounding, str) else int(rounding)
    _check("dfp_quantize_blocked", lib().dfp_quantize_blocked(rows, cols, block, bits, rnd, seed, role, _ptr(src),
                                                              _ptr(dst), _ptr(exps), _ptr(scale), _stream(stream)))


def gemm_blocked_workspace_bytes(d: GemmDesc, block_k: int) -> int:
    return int(lib().dfp_gemm_blocked_workspace_bytes(ctypes.byref(d), block_k))


def alloc_gemm_blocked_workspace(d: GemmDesc, block_k: int, device="cuda"):
    n = gemm_blocked_workspace_bytes(d, block_k)
    if n == 0:
        return None
    return torch.empty((n + 255) // 256 * 256, dtype=torch.uint8, device=device)


def dfp_gemm_blocked(d: GemmDesc, block_k, a, ea, b, eb, out, sd=None, workspace=None, partials=None, stream=None):
    for t, dt, nm in ((a, torch.int16, "a"), (b, torch.int16, "b"), (ea, torch.int8, "ea"), (eb, torch.int8, "eb"),
                      (out, torch.float32, "out"), (sd, torch.int32, "sd"), (partials, torch.int32, "partials")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_gemm_blocked", lib().dfp_gemm_blocked(ctypes.byref(d), block_k, _ptr(a), _ptr(ea), _ptr(b), _ptr(eb),
                                                      _ptr(out), _ptr(sd), wp, wn, _ptr(partials), _stream(stream)))


def make_bn_desc(n, c, hw, bits=15, rounding="nearest", eps=1e-5, seed=0) -> BnDesc:
    rnd = ROUNDING[rounding] if isinstance(rounding, str) else int(rounding)
    return BnDesc(n, c, hw, bits, rnd, eps, seed)


def bn_workspace_bytes(d: BnDesc) -> int:
    return int(lib().dfp_bn_workspace_bytes(ctypes.byref(d)))


def alloc_bn_workspace(d: BnDesc, device="cuda"):
    n = bn_workspace_bytes(d)
    return torch.empty(max(256, (n + 255) // 256 * 256), dtype=torch.uint8, device=device)


def dfp_bn_relu_fwd(d: BnDesc, y, sy, gamma, beta, zq, sz, mean, inv_std, res=None, z=None, sums=None,
                    workspace=None, stream=None):
    for t, dt, nm in ((y, torch.int16, "y"), (sy, torch.int32, "sy"), (gamma, torch.float32, "gamma"),
                      (beta, torch.float32, "beta"), (res, torch.float32, "res"), (z, torch.float32, "z"),
                      (zq, torch.int16, "zq"), (sz, torch.int32, "sz"), (mean, torch.float32, "mean"),
                      (inv_std, torch.float32, "inv_std"), (sums, torch.int64, "sums")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_bn_relu_fwd", lib().dfp_bn_relu_fwd(ctypes.byref(d), _ptr(y), _ptr(sy), _ptr(gamma), _ptr(beta),
                                                    _ptr(res), _ptr(z), _ptr(zq), _ptr(sz), _ptr(mean),
                                                    _ptr(inv_std), _ptr(sums), wp, wn, _stream(stream)))


def dfp_bn_relu_bwd(d: BnDesc, dz, sdz, y, sy, gamma, beta, mean, inv_std, dyq, sdy, dgamma, dbeta, res=None,
                    dy=None, dres=None, sums=None, workspace=None, stream=None):
    for t, dt, nm in ((dz, torch.int16, "dz"), (sdz, torch.int32, "sdz"), (y, torch.int16, "y"),
                      (sy, torch.int32, "sy"), (gamma, torch.float32, "gamma"), (beta, torch.float32, "beta"),
                      (res, torch.float32, "res"), (mean, torch.float32, "mean"),
                      (inv_std, torch.float32, "inv_std"), (dy, torch.float32, "dy"), (dyq, torch.int16, "dyq"),
                      (sdy, torch.int32, "sdy"), (dgamma, torch.float32, "dgamma"),
                      (dbeta, torch.float32, "dbeta"), (dres, torch.float32, "dres"), (sums, torch.int64, "sums")):
        _need(t, dt, nm)
    wp, wn = _ws(workspace)
    _check("dfp_bn_relu_bwd", lib().dfp_bn_relu_bwd(ctypes.byref(d), _ptr(dz), _ptr(sdz), _ptr(y), _ptr(sy),
                                                    _ptr(gamma), _ptr(beta), _ptr(res), _ptr(mean), _ptr(inv_std),
                                                    _ptr(dy), _ptr(dyq), _ptr(sdy), _ptr(dgamma), _ptr(dbeta),
                                                    _ptr(dres), _ptr(sums), wp, wn, _stream(stream)))


def dfp_sgd_quantize(lr, mu, wd, bits, rounding, seed, w, v, dw, wq, sw, stream=None):
    for t, dt, nm in ((w, torch.float32, "w"), (v, torch.float32, "v"), (dw, torch.float32, "dw"),
                      (wq, torch.int16, "wq"), (sw, torch.int32, "sw")):
        _need(t, dt, nm)
    rnd = ROUNDING[rounding] if isinstance(rounding, str) else int(rounding)
    _check("dfp_sgd_quantize", lib().dfp_sgd_quantize(w.numel(), lr, mu, wd, bits, rnd, seed, _ptr(w), _ptr(v),
                                                      _ptr(dw), _ptr(wq), _ptr(sw), _stream(stream)))


def alloc_workspace(d: Desc, direction: int, device="cuda"):
    n = workspace_bytes(d, direction)
    if n == 0:
        return None
    return torch.empty((n + 255) // 256 * 256, dtype=torch.uint8, device=device)


def profile_start(capacity: int = 100000):
    _check("dfp_profile_start", lib().dfp_profile_start(capacity))


def profile_stop(capacity: int = 100000):
    """Returns [(kernel_name, ms), ...] for every launch since profile_start."""
    ids = (ctypes.c_int32 * capacity)()
    ms = (ctypes.c_float * capacity)()
    n = lib().dfp_profile_stop(ids, ms, capacity)
    return [(lib().dfp_kernel_name(ids[i]).decode(), float(ms[i])) for i in range(n)]

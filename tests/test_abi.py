"""The C ABI contract, checked on the CPU: libdfp.so loads, exports every entry
point include/dfp.h declares, and rejects invalid arguments on the host before
any HIP call (no call here reaches a kernel launch)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dfp.h")


@pytest.fixture(scope="module")
def dl():
    from paper_1802_00930_amd import dfp
    if not os.path.exists(dfp.LIB_PATH):
        pytest.skip("libdfp.so not built")
    return dfp


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dfp_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_five_calls():
    names = declared_functions()
    for n in ("dfp_quantize", "dfp_conv_fwd", "dfp_conv_bwd_data", "dfp_conv_bwd_weights", "dfp_downconvert"):
        assert n in names


def test_every_declared_symbol_is_exported(dl):
    lib = ctypes.CDLL(dl.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_exposes_same_names(dl):
    import paper_1802_00930_amd.dfp as b
    for n in ("dfp_quantize", "dfp_conv_fwd", "dfp_conv_bwd_data", "dfp_conv_bwd_weights", "dfp_downconvert",
              "dfp_conv_fwd_i32", "dfp_conv_bwd_data_i32", "dfp_downconvert_i32", "dfp_gemm",
              "dfp_quantize_tensor", "dfp_downconvert_tensor", "dfp_bn_relu_fwd", "dfp_bn_relu_bwd",
              "dfp_sgd_quantize"):
        assert callable(getattr(b, n))


def test_desc_layout_matches_header(dl):
    # 16 int32 fields then a uint64 seed: 72 bytes with natural alignment
    assert ctypes.sizeof(dl.Desc) == 72
    assert dl.Desc.seed.offset == 64


FAKE = 1 << 20  # never dereferenced: host validation rejects these calls first


def _p(v):
    return ctypes.c_void_p(v)


def good_desc(dl, **kw):
    args = dict(n=2, c=16, h=14, w=14, k=32, r=3, s=3, stride=1, pad=1, chunk_len=16)
    args.update(kw)
    return dl.make_desc(**args)


def quant(dl, d, role=0, src=FAKE, dst=FAKE, sc=FAKE):
    return dl.lib().dfp_quantize(ctypes.byref(d) if d is not None else None, role, _p(src), _p(dst), _p(sc), None)


def fwd(dl, d, ws=None, wsn=0, x=FAKE):
    return dl.lib().dfp_conv_fwd(ctypes.byref(d), _p(x), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None,
                                 _p(ws) if ws else None, wsn, None, None)


@pytest.mark.parametrize("field,value,code", [
    ("bits", 14, 3), ("bits", 17, 3), ("rounding", 4, 3), ("rounding", -1, 3), ("chunk_len", 0, 3),
    ("seg_chunks", -1, 3), ("path", 3, 3),
    ("n", 0, 2), ("c", -1, 2), ("r", 0, 2), ("stride_h", 0, 2), ("pad_w", -1, 2), ("r", 17, 2),
])
def test_quantize_rejects(dl, field, value, code):
    d = good_desc(dl)
    setattr(d, field, value)
    assert quant(dl, d) == code


def test_quantize_null_and_role(dl):
    d = good_desc(dl)
    assert quant(dl, None) == dl.ERR_NULL
    assert quant(dl, d, src=0) == dl.ERR_NULL
    assert quant(dl, d, dst=0) == dl.ERR_NULL
    assert quant(dl, d, sc=0) == dl.ERR_NULL
    assert quant(dl, d, role=5) == dl.ERR_PARAM
    assert quant(dl, d, role=-1) == dl.ERR_PARAM


def test_quantize_alignment(dl):
    d = good_desc(dl)
    assert quant(dl, d, src=FAKE + 4) == dl.ERR_ALIGN
    assert quant(dl, d, dst=FAKE + 2) == dl.ERR_ALIGN
    assert quant(dl, d, sc=FAKE + 8) == dl.ERR_ALIGN


def test_downconvert_rejects(dl):
    d = good_desc(dl)
    f = dl.lib().dfp_downconvert
    assert f(ctypes.byref(d), dl.ROLE_X, _p(FAKE), _p(FAKE), _p(FAKE), 1, None) == dl.ERR_PARAM
    assert f(ctypes.byref(d), dl.ROLE_Y, _p(FAKE), _p(FAKE), _p(FAKE), 2, None) == dl.ERR_PARAM
    assert f(ctypes.byref(d), dl.ROLE_Y, None, _p(FAKE), _p(FAKE), 1, None) == dl.ERR_NULL
    assert f(ctypes.byref(d), dl.ROLE_DX, _p(FAKE + 4), _p(FAKE), _p(FAKE), 1, None) == dl.ERR_ALIGN


def test_conv_rejects(dl):
    d = good_desc(dl)
    assert fwd(dl, d, x=0) == dl.ERR_NULL
    bad = good_desc(dl, chunk_len=0)
    assert fwd(dl, bad) == dl.ERR_PARAM
    bad = good_desc(dl, h=2, pad=0)
    assert fwd(dl, bad) == dl.ERR_SHAPE
    lib = dl.lib()
    # backward-weights with NULL dw
    assert lib.dfp_conv_bwd_weights(ctypes.byref(d), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None, None, 0,
                                    None, None) == dl.ERR_NULL
    assert lib.dfp_conv_bwd_data(ctypes.byref(bad), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None,
                                 None, 0, None, None) == dl.ERR_SHAPE


def test_conv_workspace_checked(dl):
    for direction in (dl.FWD, dl.BWD_DATA, dl.BWD_WT):
        d = good_desc(dl, path=dl.PATH_MFMA, chunk_len=64)
        need = dl.workspace_bytes(d, direction)
        if need == 0:
            continue
        lib = dl.lib()
        args_small = (_p(FAKE), need - 1)
        if direction == dl.FWD:
            rc = lib.dfp_conv_fwd(ctypes.byref(d), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None,
                                  *args_small, None, None)
        elif direction == dl.BWD_DATA:
            rc = lib.dfp_conv_bwd_data(ctypes.byref(d), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None,
                                       *args_small, None, None)
        else:
            rc = lib.dfp_conv_bwd_weights(ctypes.byref(d), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE),
                                          *args_small, None, None)
        assert rc == dl.ERR_WORKSPACE


def _conv_i32(dl, direction, d, so=FAKE, ws=None, wsn=0):
    f = dl.lib().dfp_conv_fwd_i32 if direction == dl.FWD else dl.lib().dfp_conv_bwd_data_i32
    return f(ctypes.byref(d), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(so) if so else None,
             _p(ws) if ws else None, wsn, None)


def test_conv_i32_rejects(dl):
    # the single chunk must cover the reduction: C*R*S = 144 forward, K*R*S = 288 backward-data
    for direction, t in ((dl.FWD, 144), (dl.BWD_DATA, 288)):
        short = good_desc(dl, chunk_len=t - 1, path=dl.PATH_VALU)
        assert _conv_i32(dl, direction, short) == dl.ERR_PARAM
        ok = good_desc(dl, chunk_len=t, path=dl.PATH_VALU)
        assert _conv_i32(dl, direction, ok, so=0) == dl.ERR_NULL
        assert _conv_i32(dl, direction, ok, so=FAKE + 8) == dl.ERR_ALIGN
        mf = good_desc(dl, chunk_len=t, path=dl.PATH_MFMA)
        need = dl.workspace_bytes(mf, direction)
        assert need > 0
        assert _conv_i32(dl, direction, mf, ws=FAKE, wsn=need - 1) == dl.ERR_WORKSPACE
    assert _conv_i32(dl, dl.FWD, good_desc(dl, chunk_len=144, h=2, pad=0)) == dl.ERR_SHAPE


def test_downconvert_i32_rejects(dl):
    d = good_desc(dl)
    f = dl.lib().dfp_downconvert_i32

    def call(role=dl.ROLE_Y, src=FAKE, sin=FAKE, dst=FAKE + 4096, sout=FAKE + 8192, ready=1):
        return f(ctypes.byref(d), role, _p(src), _p(sin), _p(dst), _p(sout), ready, None)
    assert call(role=dl.ROLE_X) == dl.ERR_PARAM
    assert call(role=dl.ROLE_W) == dl.ERR_PARAM
    assert call(ready=2) == dl.ERR_PARAM
    assert call(sout=FAKE) == dl.ERR_PARAM  # sin and sout must differ
    assert call(src=0) == dl.ERR_NULL
    assert call(sin=0) == dl.ERR_NULL
    assert call(src=FAKE + 8) == dl.ERR_ALIGN
    assert call(dst=FAKE + 4096 + 4) == dl.ERR_ALIGN
    assert call(sin=FAKE + 4) == dl.ERR_ALIGN


def test_gemm_desc_layout(dl):
    assert ctypes.sizeof(dl.GemmDesc) == 32


def _gemm(dl, d, a=FAKE, b=FAKE + 4096, out=FAKE + 8192, sd=None, ws=None, wsn=0, parts=None):
    return dl.lib().dfp_gemm(ctypes.byref(d) if d is not None else None, _p(a), _p(FAKE), _p(b), _p(FAKE),
                             _p(out), _p(sd) if sd else None, _p(ws) if ws else None, wsn,
                             _p(parts) if parts else None, None)


def test_gemm_rejects(dl):
    ok = dict(m=64, n=1000, k=2048, trans_b=True, chunk_len=64, path=dl.PATH_VALU)
    assert _gemm(dl, None) == dl.ERR_NULL
    for field, value, code in (("m", 0, dl.ERR_SHAPE), ("k", -1, dl.ERR_SHAPE), ("trans_a", 2, dl.ERR_PARAM),
                               ("chunk_len", 0, dl.ERR_PARAM), ("bits", 14, dl.ERR_PARAM),
                               ("path", 3, dl.ERR_PARAM)):
        d = dl.make_gemm_desc(**ok)
        setattr(d, field, value)
        assert _gemm(dl, d) == code, field
    big = dl.make_gemm_desc(**dict(ok, m=2 ** 21, n=2 ** 20))
    assert _gemm(dl, big) == dl.ERR_SHAPE  # m*n > 2^40
    d = dl.make_gemm_desc(**ok)
    assert _gemm(dl, d, a=0) == dl.ERR_NULL
    assert _gemm(dl, d, out=0) == dl.ERR_NULL
    assert _gemm(dl, d, a=FAKE + 1) == dl.ERR_ALIGN
    assert _gemm(dl, d, out=FAKE + 8192 + 2) == dl.ERR_ALIGN
    assert _gemm(dl, d, sd=FAKE + 8) == dl.ERR_ALIGN
    assert dl.gemm_workspace_bytes(d) == 0  # VALU path needs none
    mf = dl.make_gemm_desc(**dict(ok, path=dl.PATH_MFMA))
    need = dl.gemm_workspace_bytes(mf)
    # A digits 32*2 x 64 rows x 64 B, B digits 1000 columns x 128 groups x 32 B, 64 block offsets
    assert need == 64 * 64 * 64 + 1000 * 128 * 32 + 512
    assert _gemm(dl, mf, ws=FAKE, wsn=need - 1) == dl.ERR_WORKSPACE
    assert _gemm(dl, mf, ws=FAKE + 128, wsn=need) == dl.ERR_WORKSPACE
    assert dl.gemm_num_chunks(mf) == 32
    assert dl.gemm_num_chunks(dl.make_gemm_desc(**dict(ok, chunk_len=0))) == -1
    assert dl.gemm_workspace_bytes(dl.make_gemm_desc(**dict(ok, bits=16, path=dl.PATH_AUTO))) == 0


def test_flat_quantize_rejects(dl):
    q, dc = dl.lib().dfp_quantize_tensor, dl.lib().dfp_downconvert_tensor
    good = (1000, 15, 0, 0, dl.ROLE_X)
    assert q(*good, None, _p(FAKE), _p(FAKE), None) == dl.ERR_NULL
    assert q(0, 15, 0, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert q(1000, 14, 0, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert q(1000, 15, 4, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert q(1000, 15, 0, 0, 5, _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert q(*good, _p(FAKE + 4), _p(FAKE), _p(FAKE), None) == dl.ERR_ALIGN
    assert dc(*good, _p(FAKE), _p(FAKE), _p(FAKE), 2, None) == dl.ERR_PARAM
    assert dc(*good, _p(FAKE), _p(FAKE + 2), _p(FAKE), 1, None) == dl.ERR_ALIGN


def test_blocked_rejects(dl):
    lib = dl.lib()
    d = dl.make_gemm_desc(64, 1000, 2048, False, True, chunk_len=64)

    def g(desc, bk=128, a=FAKE, ea=FAKE + 4096, ws=None, wsn=0):
        return lib.dfp_gemm_blocked(ctypes.byref(desc), bk, _p(a), _p(ea), _p(FAKE + 8192), _p(FAKE + 12288),
                                    _p(FAKE + 16384), None, _p(ws) if ws else None, wsn, None, None)
    assert g(d, bk=96) == dl.ERR_PARAM      # block not a multiple of the chunk
    assert g(d, bk=0) == dl.ERR_PARAM
    assert g(dl.make_gemm_desc(64, 1000, 2048, True, True, chunk_len=64)) == dl.ERR_PARAM
    assert g(dl.make_gemm_desc(64, 1000, 2048, False, False, chunk_len=64)) == dl.ERR_PARAM
    assert g(d, ea=0) == dl.ERR_NULL
    assert g(d, a=FAKE + 1) == dl.ERR_ALIGN
    need = dl.gemm_blocked_workspace_bytes(d, 128)
    assert need == dl.gemm_workspace_bytes(d) > 0
    assert g(d, ws=FAKE, wsn=need - 1) == dl.ERR_WORKSPACE
    # more than 80 exponent blocks, P = 16 or a chunk not a multiple of 32: VALU path, no workspace
    assert dl.gemm_blocked_workspace_bytes(d, 16 * 1) == 0
    assert dl.gemm_blocked_workspace_bytes(dl.make_gemm_desc(64, 1000, 2048, False, True, 64, bits=16), 128) == 0
    assert dl.gemm_blocked_workspace_bytes(dl.make_gemm_desc(64, 1000, 2048, False, True, 16), 128) == 0
    q = lib.dfp_quantize_blocked
    assert q(0, 10, 4, 15, 0, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_SHAPE
    assert q(3, 10, 0, 15, 0, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert q(3, 10, 4, 17, 0, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert q(3, 10, 4, 15, 0, 0, 0, _p(FAKE), _p(FAKE), None, _p(FAKE), None) == dl.ERR_NULL
    assert q(3, 10, 4, 15, 0, 0, 0, _p(FAKE + 2), _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_ALIGN


def test_bn_desc_layout(dl):
    # five int32, a float, then the uint64 seed at offset 24
    assert ctypes.sizeof(dl.BnDesc) == 32
    assert dl.BnDesc.seed.offset == 24


def test_bn_rejects(dl):
    lib = dl.lib()
    d = dl.make_bn_desc(32, 64, 3136)
    need = dl.bn_workspace_bytes(d)
    # 32 image splits x 64 channels x 24 B of partial sums, then 64 x 16 B of coefficients
    assert need == 32 * 64 * 24 + 1024

    def f(desc, y=FAKE, zq=FAKE + 4096, res=None, z=None, ws=FAKE + 65536, wsn=need, gamma=FAKE):
        return lib.dfp_bn_relu_fwd(ctypes.byref(desc) if desc is not None else None, _p(y), _p(FAKE), _p(gamma),
                                   _p(FAKE), _p(res) if res else None, _p(z) if z else None, _p(zq), _p(FAKE),
                                   _p(FAKE), _p(FAKE), None, _p(ws) if ws else None, wsn, None)
    assert f(None) == dl.ERR_NULL
    assert f(d, gamma=0) == dl.ERR_NULL
    for field, value, code in (("n", 0, dl.ERR_SHAPE), ("hw", -3, dl.ERR_SHAPE), ("bits", 14, dl.ERR_PARAM),
                               ("rounding", 4, dl.ERR_PARAM), ("eps", -1e-5, dl.ERR_PARAM),
                               ("eps", float("nan"), dl.ERR_PARAM), ("eps", float("inf"), dl.ERR_PARAM)):
        bad = dl.make_bn_desc(32, 64, 3136)
        setattr(bad, field, value)
        assert f(bad) == code, field
    assert f(dl.make_bn_desc(2 ** 11, 2 ** 10, 2 ** 10)) == dl.ERR_SHAPE  # 2^31 elements
    assert dl.bn_workspace_bytes(dl.make_bn_desc(0, 64, 3136)) == 0
    assert f(d, y=FAKE + 8) == dl.ERR_ALIGN
    assert f(d, res=FAKE + 4) == dl.ERR_ALIGN
    assert f(d, z=FAKE + 4) == dl.ERR_ALIGN
    assert f(d, ws=None) == dl.ERR_WORKSPACE
    assert f(d, wsn=need - 1) == dl.ERR_WORKSPACE
    assert f(d, ws=FAKE + 65536 + 128) == dl.ERR_WORKSPACE

    def b(desc, dz=FAKE, dyq=FAKE + 4096, dgamma=FAKE, wsn=need):
        return lib.dfp_bn_relu_bwd(ctypes.byref(desc), _p(dz), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None,
                                   _p(FAKE), _p(FAKE), None, _p(dyq), _p(FAKE), _p(dgamma), _p(FAKE), None, None,
                                   _p(FAKE + 65536), wsn, None)
    assert b(d, dgamma=0) == dl.ERR_NULL
    assert b(d, dz=FAKE + 2) == dl.ERR_ALIGN
    assert b(d, wsn=0) == dl.ERR_WORKSPACE
    s = lib.dfp_sgd_quantize
    assert s(1000, 0.1, 0.9, 1e-4, 15, 0, 0, _p(FAKE), _p(FAKE), None, _p(FAKE), _p(FAKE), None) == dl.ERR_NULL
    assert s(0, 0.1, 0.9, 1e-4, 15, 0, 0, _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert s(1000, 0.1, 0.9, 1e-4, 16, 5, 0, _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE), None) == dl.ERR_PARAM
    assert s(1000, 0.1, 0.9, 1e-4, 15, 0, 0, _p(FAKE + 4), _p(FAKE), _p(FAKE), _p(FAKE), _p(FAKE),
             None) == dl.ERR_ALIGN


def test_host_queries(dl):
    d = good_desc(dl, chunk_len=16)
    assert dl.output_dims(d) == (14, 14)
    assert dl.num_chunks(d, dl.FWD) == 9      # 16*9 = 144 products / 16
    assert dl.num_chunks(d, dl.BWD_DATA) == 18  # 32*9 = 288 / 16
    assert dl.num_chunks(d, dl.BWD_WT) == 25  # 2*14*14 = 392 / 16 -> 24.5
    s = good_desc(dl, h=9, w=8, stride=2, pad=1)
    assert dl.output_dims(s) == (5, 4)
    assert dl.num_chunks(good_desc(dl, chunk_len=0), dl.FWD) == -1
    for code in range(8):
        assert isinstance(dl.status_str(code), str)
    assert dl.lib().dfp_kernel_name(0) == b"scale_reset"


def test_oracle_not_reachable_from_product():
    """The product package never imports the oracle."""
    pkg = os.path.join(ROOT, "paper_1802_00930_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "import oracle" not in text and "from oracle" not in text, fn
                assert "liboracle" not in text and "dfp_oracle" not in text, fn


def test_noalloc_scratch_limit_and_nulls_on_host(dl):
    """dfp_conv_bwd_weights_noalloc rejects, before any HIP call, null
    operands and a layer whose workspace exceeds the static scratch."""
    lib = dl.lib()
    big = dl.make_desc(32, 64, 224, 224, 64, 3, 3, 1, 1, chunk_len=64, seg_chunks=16)
    assert dl.workspace_bytes(big, dl.BWD_WT) > dl.NOALLOC_SCRATCH_BYTES
    args = [_p(FAKE)] * 5
    assert lib.dfp_conv_bwd_weights_noalloc(ctypes.byref(big), *args, None) == dl.ERR_SCRATCH_LIMIT
    small = good_desc(dl)
    assert lib.dfp_conv_bwd_weights_noalloc(ctypes.byref(small), None, *args[1:], None) == dl.ERR_NULL
    bad = good_desc(dl, bits=14)
    assert lib.dfp_conv_bwd_weights_noalloc(ctypes.byref(bad), *args, None) == dl.ERR_PARAM
    assert "64 MiB" in dl.status_str(dl.ERR_SCRATCH_LIMIT)

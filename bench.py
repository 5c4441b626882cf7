#!/usr/bin/env python3
"""Benchmark of the DFP INT16 convolution hot path on one MI355X.

One step = the whole path over one batch of the ResNet-50 conv2_x 3x3 layer
(N=32, C=K=64, 56x56, 3x3, stride 1, pad 1; ReLU(N(0,1)) activations,
He-normal weights, output gradients N(0,1)*1e-3; stochastic rounding, seed 1;
DFP15; chunk length 64):

    Q(x), Q(w), Q(dy)             quantise FP32 -> DFP16      (Eq. 1-3)
    fwd, DC(y)                    forward conv, down-convert  (Alg. 2, Sec. 4.3)
    bwd-data, DC(dx)              backward-data, down-convert
    bwd-wt                        backward-weights (FP32 dW)

value = algorithmic INT16 operations of the three convolutions
(3 x 2 x N*K*C*R*S*P*Q) per second of whole-step time, inputs resident in HBM.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DFP INT16 conv TOPS (fwd/bwd-data/bwd-wt) and % of integer-path roofline"
WORKLOAD = "resnet50_conv2x_3x3"
# MI355X published peaks used for the roofline fraction.
PEAK_INT8_MFMA_TOPS = 5030.0          # dense int8 MFMA, 256 CU x 2.4 GHz x 8192 ops/clk
PEAK_INT16_BYTESPLIT_TOPS = PEAK_INT8_MFMA_TOPS / 4  # 4 int8 products per INT16 product
PEAK_VALU_DOT2_TOPS = 157.3           # 256 CU x 4 SIMD x 16 lanes x 2.4 GHz x 4 ops (dot2)
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--chunk", type=int, default=64)
    ap.add_argument("--path", type=int, default=0, help="0 auto, 1 MFMA, 2 VALU")
    ap.add_argument("--seg-chunks", type=int, default=16,
                    help="backward-weights segment size G in chunks (part of the numerics: the oracle uses the same)")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-dfp32", action="store_true", help="skip the DFP-32-output variant of the step")
    ap.add_argument("--no-gemm", action="store_true", help="skip the GEMM measurements")
    ap.add_argument("--no-train-ops", action="store_true", help="skip the BN / SGD measurements")
    ap.add_argument("--no-layers", action="store_true",
                    help="skip the per-layer sweep (ResNet-50 conv4_x 1x1 pair, VGG-16 conv1_2 / conv3_3, all 53 "
                         "ResNet-50 convolutions)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--detail-out", default="", metavar="PATH",
                    help="also write every detail block and the headline line to this file")
    ap.add_argument("--peaks", action="store_true",
                    help="only measure the unit ceilings (int8 MFMA, v_dot2_i32_i16, the byte-split chunk loop with "
                         "register operands, HBM read and copy) with libpeaks.so")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES five times (counter calibration)")
    return ap.parse_args()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` (one of the three convolution
    directions) from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE passes
    (calibrated on a plain copy), or None when none was taken on that kernel
    or its source has changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_conv2x_3x3.json")
    try:
        recs = json.load(open(path))["records"]
    except (OSError, ValueError, KeyError):
        return None
    for rec in recs:
        if rec.get("kernel") != kernel:
            continue
        try:
            src = open(os.path.join(ROOT, rec["source"]), "rb").read()
        except (OSError, KeyError):
            return None
        if hashlib.sha256(src).hexdigest() != rec.get("source_sha256"):
            return None
        return {"bytes": int(rec["fetch_bytes"] + rec["write_bytes"]), "fetch_bytes": int(rec["fetch_bytes"]),
                "write_bytes": int(rec["write_bytes"]), "device_kernel": rec.get("device_kernel"),
                "source": rec.get("summary")}
    return None


def copy_probe(nbytes):
    """A plain copy kernel of known size: its FETCH_SIZE / WRITE_SIZE counters
    calibrate the byte counts of the DFP kernels (rocprofv3 --pmc)."""
    import torch
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "launches": 5}), flush=True)


def measure_peaks():
    """Measured ceilings next to the published ones: each kernel runs twice
    and the second launch is timed (HIP events)."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_1802_00930_amd", "libpeaks.so")
    if not os.path.exists(path):
        raise ImportError("libpeaks.so is not built; run __graft_entry__.build()")
    torch.cuda.init()
    lib = ctypes.CDLL(path)
    for fn, args in (("peaks_mfma_i8", [ctypes.c_int] * 3), ("peaks_dot2_i16", [ctypes.c_int] * 2),
                     ("peaks_chunk_loop", [ctypes.c_int] * 2), ("peaks_hbm_read", [ctypes.c_int64, ctypes.c_int]),
                     ("peaks_hbm_copy", [ctypes.c_int64, ctypes.c_int])):
        getattr(lib, fn).argtypes = args
        getattr(lib, fn).restype = ctypes.c_float
    res = {}
    blocks, iters = 1024, 20000  # 4 waves per SIMD on 256 CUs
    for shape, name in ((0, "mfma_i32_32x32x32_i8"), (1, "mfma_i32_16x16x64_i8")):
        ms = lib.peaks_mfma_i8(shape, blocks, iters)
        ops = blocks * 4 * iters * 4 * 32768 * 2.0
        res[name] = {"ms": round(ms, 4), "int8_tops": round(ops / ms / 1e9, 1),
                     "frac_of_published": round(ops / ms / 1e9 / PEAK_INT8_MFMA_TOPS, 4)}
    dblocks, diters = 2048, 20000
    ms = lib.peaks_dot2_i16(dblocks, diters)
    ops = dblocks * 256 * 8 * diters * 2 * 2.0
    res["dot2_i32_i16"] = {"ms": round(ms, 4), "int16_tops": round(ops / ms / 1e9, 1),
                           "frac_of_assumed_full_rate": round(ops / ms / 1e9 / PEAK_VALU_DOT2_TOPS, 4)}
    citers = 5000
    ms = lib.peaks_chunk_loop(blocks, citers)
    ops = blocks * 4 * citers * 32 * 32 * 64 * 2.0
    res["bytesplit_chunk_loop_l64"] = {"ms": round(ms, 4), "int16_eq_tops": round(ops / ms / 1e9, 1),
                                       "frac_of_bytesplit_peak": round(ops / ms / 1e9 / PEAK_INT16_BYTESPLIT_TOPS, 4)}
    nbytes = 1 << 30
    ms = lib.peaks_hbm_read(nbytes, 2048)
    res["hbm_read_1GiB"] = {"ms": round(ms, 4), "gbs": round(nbytes / ms / 1e6, 1),
                            "frac_of_published": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4)}
    ms = lib.peaks_hbm_copy(nbytes // 2, 2048)
    res["hbm_copy_512MiB"] = {"ms": round(ms, 4), "gbs_read_plus_write": round(nbytes / ms / 1e6, 1),
                              "frac_of_published": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4)}
    print(json.dumps({"peaks": res}), flush=True)


class Step:
    """Device buffers and the ABI calls of one step."""

    def __init__(self, layer, x, w, dy, L, rounding, seed, path, dev, G=0, bwd_data=True):
        import torch
        from paper_1802_00930_amd import dfp
        self.bwd_data = bwd_data  # False: the network's first layer, whose input gradient training never uses
        self.dfp = dfp
        self.torch = torch
        self.layer = layer
        self.d = dfp.make_desc(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride,
                               layer.pad, chunk_len=L, seg_chunks=G, rounding=rounding, seed=seed, path=path)
        self.fx, self.fw, self.fdy = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
        self.qx = torch.empty_like(self.fx, dtype=torch.int16)
        self.qw = torch.empty_like(self.fw, dtype=torch.int16)
        self.qdy = torch.empty_like(self.fdy, dtype=torch.int16)
        self.y = torch.empty(layer.n, layer.k, layer.p, layer.q, dtype=torch.float32, device=dev)
        self.dx = torch.empty_like(self.fx)
        self.dw = torch.empty_like(self.fw)
        self.qy = torch.empty_like(self.y, dtype=torch.int16)
        self.qdx = torch.empty_like(self.dx, dtype=torch.int16)
        self.sx, self.sw, self.sdy, self.sy, self.sdx = (dfp.new_scale(dev) for _ in range(5))
        self.ws = [dfp.alloc_workspace(self.d, k, dev) for k in range(3)]

    def run(self):
        dfp, d = self.dfp, self.d
        dfp.dfp_quantize(d, dfp.ROLE_X, self.fx, self.qx, self.sx)
        dfp.dfp_quantize(d, dfp.ROLE_W, self.fw, self.qw, self.sw)
        dfp.dfp_quantize(d, dfp.ROLE_DY, self.fdy, self.qdy, self.sdy)
        dfp.dfp_conv_fwd(d, self.qx, self.sx, self.qw, self.sw, self.y, self.sy, self.ws[0])
        dfp.dfp_downconvert(d, dfp.ROLE_Y, self.y, self.qy, self.sy, amax_ready=True)
        if self.bwd_data:
            dfp.dfp_conv_bwd_data(d, self.qdy, self.sdy, self.qw, self.sw, self.dx, self.sdx, self.ws[1])
            dfp.dfp_downconvert(d, dfp.ROLE_DX, self.dx, self.qdx, self.sdx, amax_ready=True)
        dfp.dfp_conv_bwd_weights(d, self.qx, self.sx, self.qdy, self.sdy, self.dw, self.ws[2])


class StepDfp32(Step):
    """The same step with forward and backward-data emitting single-chunk
    DFP-32 outputs (chunk = the whole reduction, INT32 with exponent Ea + Eb)
    and the integer down-convert of Eq. 6 taking the epilogue's max."""

    def __init__(self, layer, x, w, dy, L, rounding, seed, path, dev, G=0):
        super().__init__(layer, x, w, dy, L, rounding, seed, path, dev, G)
        dfp, torch = self.dfp, self.torch
        T = max(layer.c, layer.k) * layer.r * layer.s
        self.d32 = dfp.make_desc(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride,
                                 layer.pad, chunk_len=T, rounding=rounding, seed=seed, path=path)
        self.y = self.y.view(torch.int32)
        self.dx = self.dx.view(torch.int32)
        self.ws32 = [dfp.alloc_workspace(self.d32, k, dev) for k in range(2)]
        self.sqy, self.sqdx = dfp.new_scale(dev), dfp.new_scale(dev)

    def run(self):
        dfp, d, d32 = self.dfp, self.d, self.d32
        dfp.dfp_quantize(d, dfp.ROLE_X, self.fx, self.qx, self.sx)
        dfp.dfp_quantize(d, dfp.ROLE_W, self.fw, self.qw, self.sw)
        dfp.dfp_quantize(d, dfp.ROLE_DY, self.fdy, self.qdy, self.sdy)
        dfp.dfp_conv_fwd_i32(d32, self.qx, self.sx, self.qw, self.sw, self.y, self.sy, self.ws32[0])
        dfp.dfp_downconvert_i32(d32, dfp.ROLE_Y, self.y, self.sy, self.qy, self.sqy, amax_ready=True)
        dfp.dfp_conv_bwd_data_i32(d32, self.qdy, self.sdy, self.qw, self.sw, self.dx, self.sdx, self.ws32[1])
        dfp.dfp_downconvert_i32(d32, dfp.ROLE_DX, self.dx, self.sdx, self.qdx, self.sqdx, amax_ready=True)
        dfp.dfp_conv_bwd_weights(d, self.qx, self.sx, self.qdy, self.sdy, self.dw, self.ws[2])


class FcStep:
    """One DFP step of a fully connected layer through the GEMM entry point:
    Q(x), Q(W), Q(dy), y = x W^T, DC(y), dx = dy W, DC(dx), dW = dy^T x."""

    def __init__(self, batch, fin, fout, L, rounding, seed, dev):
        import torch
        from paper_1802_00930_amd import dfp
        self.dfp, self.torch = dfp, torch
        self.rounding, self.seed = rounding, seed
        g = torch.Generator(device="cpu").manual_seed(seed)
        self.fx = torch.relu(torch.randn(batch, fin, generator=g)).to(dev)
        self.fw = (torch.randn(fout, fin, generator=g) * (1.0 / fin) ** 0.5).to(dev)
        self.fdy = (torch.randn(batch, fout, generator=g) * 1e-3).to(dev)
        self.q = {k: torch.empty_like(v, dtype=torch.int16) for k, v in
                  (("x", self.fx), ("w", self.fw), ("dy", self.fdy))}
        self.s = {k: dfp.new_scale(dev) for k in ("x", "w", "dy", "y", "dx")}
        self.y = torch.empty(batch, fout, device=dev)
        self.dx = torch.empty(batch, fin, device=dev)
        self.dw = torch.empty(fout, fin, device=dev)
        self.qy = torch.empty_like(self.y, dtype=torch.int16)
        self.qdx = torch.empty_like(self.dx, dtype=torch.int16)
        self.d = [dfp.make_gemm_desc(batch, fout, fin, False, True, L),
                  dfp.make_gemm_desc(batch, fin, fout, False, False, L),
                  dfp.make_gemm_desc(fout, fin, batch, True, False, L)]
        self.ws = [dfp.alloc_gemm_workspace(d, dev) for d in self.d]
        self.macs = batch * fin * fout

    def run(self):
        dfp, q, s, r, sd = self.dfp, self.q, self.s, self.rounding, self.seed
        dfp.dfp_quantize_tensor(15, r, sd, dfp.ROLE_X, self.fx, q["x"], s["x"])
        dfp.dfp_quantize_tensor(15, r, sd, dfp.ROLE_W, self.fw, q["w"], s["w"])
        dfp.dfp_quantize_tensor(15, r, sd, dfp.ROLE_DY, self.fdy, q["dy"], s["dy"])
        dfp.dfp_gemm(self.d[0], q["x"], s["x"], q["w"], s["w"], self.y, s["y"], self.ws[0])
        dfp.dfp_downconvert_tensor(15, r, sd, dfp.ROLE_Y, self.y, self.qy, s["y"], amax_ready=True)
        dfp.dfp_gemm(self.d[1], q["dy"], s["dy"], q["w"], s["w"], self.dx, s["dx"], self.ws[1])
        dfp.dfp_downconvert_tensor(15, r, sd, dfp.ROLE_DX, self.dx, self.qdx, s["dx"], amax_ready=True)
        dfp.dfp_gemm(self.d[2], q["dy"], s["dy"], q["x"], s["x"], self.dw, None, self.ws[2])


class GemmStep:
    """One DFP16 GEMM D = A B^T of m x n x k on operands already quantised."""

    def __init__(self, m, n, k, L, dev):
        import torch
        from paper_1802_00930_amd import dfp
        self.dfp, self.torch = dfp, torch
        g = torch.Generator(device="cpu").manual_seed(7)
        self.a = torch.randint(-16384, 16385, (m, k), dtype=torch.int16, generator=g).to(dev)
        self.b = torch.randint(-16384, 16385, (n, k), dtype=torch.int16, generator=g).to(dev)
        self.sa, self.sb, self.sd = (torch.tensor([0, -14, 0, 0], dtype=torch.int32, device=dev) for _ in range(3))
        self.out = torch.empty(m, n, device=dev)
        self.d = dfp.make_gemm_desc(m, n, k, False, True, L)
        self.ws = dfp.alloc_gemm_workspace(self.d, dev)
        self.macs = m * n * k

    def run(self):
        self.dfp.dfp_gemm(self.d, self.a, self.sa, self.b, self.sb, self.out, self.sd, self.ws)


class BlockedFcStep:
    """Blocked-DFP forward of the FC layer: x and W quantised per block of bk
    input features, y = x W^T with per-chunk block scales."""

    def __init__(self, batch, fin, fout, L, bk, rounding, seed, dev):
        import torch
        from paper_1802_00930_amd import dfp
        self.dfp, self.torch = dfp, torch
        self.rounding, self.seed, self.bk = rounding, seed, bk
        g = torch.Generator(device="cpu").manual_seed(seed)
        self.fx = torch.relu(torch.randn(batch, fin, generator=g)).to(dev)
        self.fw = (torch.randn(fout, fin, generator=g) * (1.0 / fin) ** 0.5).to(dev)
        nb = (fin + bk - 1) // bk
        self.qx = torch.empty_like(self.fx, dtype=torch.int16)
        self.qw = torch.empty_like(self.fw, dtype=torch.int16)
        self.ex = torch.empty(nb, batch, dtype=torch.int8, device=dev)
        self.ew = torch.empty(nb, fout, dtype=torch.int8, device=dev)
        self.sx, self.sw, self.sy = (dfp.new_scale(dev) for _ in range(3))
        self.y = torch.empty(batch, fout, device=dev)
        self.d = dfp.make_gemm_desc(batch, fout, fin, False, True, L)
        self.ws = dfp.alloc_gemm_blocked_workspace(self.d, bk, dev)
        self.macs = batch * fin * fout

    def run(self):
        dfp, r, sd = self.dfp, self.rounding, self.seed
        dfp.dfp_quantize_blocked(self.bk, 15, r, sd, dfp.ROLE_X, self.fx, self.qx, self.ex, self.sx)
        dfp.dfp_quantize_blocked(self.bk, 15, r, sd, dfp.ROLE_W, self.fw, self.qw, self.ew, self.sw)
        dfp.dfp_gemm_blocked(self.d, self.bk, self.qx, self.ex, self.qw, self.ew, self.y, self.sy, self.ws)


class BlockedGemmStep(GemmStep):
    """GemmStep with per-block exponents (block of bk reduction indices)."""

    def __init__(self, m, n, k, L, bk, dev):
        super().__init__(m, n, k, L, dev)
        import torch
        nb = (k + bk - 1) // bk
        g = torch.Generator(device="cpu").manual_seed(8)
        self.bk = bk
        self.ea = torch.randint(-20, -10, (nb, m), dtype=torch.int8, generator=g).to(dev)
        self.eb = torch.randint(-20, -10, (nb, n), dtype=torch.int8, generator=g).to(dev)
        self.ws = self.dfp.alloc_gemm_blocked_workspace(self.d, bk, dev)

    def run(self):
        self.dfp.dfp_gemm_blocked(self.d, self.bk, self.a, self.ea, self.b, self.eb, self.out, self.sd, self.ws)


class TrainOpsStep:
    """The steps either side of the layer's convolutions: BN + ReLU forward on
    the DFP16 conv output with Q_a, its backward with Q_e, and FP32 SGD with
    Q_w on the layer's weights (one call each)."""

    def __init__(self, layer, rounding, seed, dev):
        import torch
        from paper_1802_00930_amd import dfp
        self.dfp, self.torch = dfp, torch
        n, c, hw = layer.n, layer.k, layer.p * layer.q
        g = torch.Generator(device="cpu").manual_seed(seed)
        self.d = dfp.make_bn_desc(n, c, hw, rounding=rounding, seed=seed)
        self.y = torch.randint(-16384, 16385, (n, c, hw), dtype=torch.int16, generator=g).to(dev)
        self.dz = torch.randint(-16384, 16385, (n, c, hw), dtype=torch.int16, generator=g).to(dev)
        self.sy = torch.tensor([0, -12, 0, 0], dtype=torch.int32, device=dev)
        self.sdz = torch.tensor([0, -24, 0, 0], dtype=torch.int32, device=dev)
        self.gamma = (torch.rand(c, generator=g) + 0.5).to(dev)
        self.beta = (torch.rand(c, generator=g) - 0.5).to(dev)
        self.zq = torch.empty_like(self.y)
        self.dyq = torch.empty_like(self.y)
        self.sz, self.sdy, self.swq = (dfp.new_scale(dev) for _ in range(3))
        self.mean = torch.empty(c, device=dev)
        self.inv = torch.empty(c, device=dev)
        self.dg = torch.empty(c, device=dev)
        self.db = torch.empty(c, device=dev)
        self.ws = dfp.alloc_bn_workspace(self.d, dev)
        nw = layer.k * layer.c * layer.r * layer.s
        self.w = (torch.randn(nw, generator=g) * 0.05).to(dev)
        self.v = torch.zeros(nw, device=dev)
        self.dw = (torch.randn(nw, generator=g) * 1e-3).to(dev)
        self.wq = torch.empty(nw, dtype=torch.int16, device=dev)
        self.elems, self.nw = n * c * hw, nw
        self.rounding, self.seed = rounding, seed

    def run(self):
        dfp = self.dfp
        dfp.dfp_bn_relu_fwd(self.d, self.y, self.sy, self.gamma, self.beta, self.zq, self.sz, self.mean, self.inv,
                            workspace=self.ws)
        dfp.dfp_bn_relu_bwd(self.d, self.dz, self.sdz, self.y, self.sy, self.gamma, self.beta, self.mean, self.inv,
                            self.dyq, self.sdy, self.dg, self.db, workspace=self.ws)
        dfp.dfp_sgd_quantize(1e-3, 0.9, 1e-4, 15, self.rounding, self.seed, self.w, self.v, self.dw, self.wq,
                             self.swq)


def kernel_table(recs, steps):
    per = {}
    for name, ms in recs:
        per.setdefault(name, []).append(ms)
    return {k: {"launches_per_step": len(v) / steps, "avg_ms": round(float(np.mean(v)), 5)} for k, v in per.items()}


def timed(step, steps, warmup, profile=False):
    """Seconds per step over `steps` steps after `warmup` untimed ones.  With
    profile=True every library launch is bracketed by HIP events on its stream
    and the per-launch durations are returned too."""
    torch = step.torch
    for _ in range(warmup):
        step.run()
    torch.cuda.synchronize()
    if profile:
        step.dfp.profile_start(64 * steps + 64)
    t0 = time.perf_counter()
    for _ in range(steps):
        step.run()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    recs = step.dfp.profile_stop(64 * steps + 64) if profile else []
    return (t1 - t0) / steps, recs


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _omp():
    """libgomp as loaded by the oracle (its thread count is set per call site)."""
    import ctypes
    lib = ctypes.CDLL("libgomp.so.1")
    lib.omp_get_max_threads.restype = ctypes.c_int
    lib.omp_set_num_threads.argtypes = [ctypes.c_int]
    return lib


def cpu_baseline(layer, x, w, dy, L, G, rounding, seed, budget_s):
    """The CPU oracle on a bounded sample of the same layer: every quantisation
    in full, then the three convolutions at sampled output elements, once on
    all host threads and once on one thread (a third of the budget)."""
    import oracle
    oracle.lib()
    omp = _omp()
    threads = int(omp.omp_get_max_threads())
    rnd = oracle.ROUNDING[rounding]
    t0 = time.perf_counter()
    ox, ex, _ = oracle.quantize(x, 15, rnd, seed, oracle.ROLE_X)
    ow, ew, _ = oracle.quantize(w, 15, rnd, seed, oracle.ROLE_W)
    ody, edy, _ = oracle.quantize(dy, 15, rnd, seed, oracle.ROLE_DY)
    tq = time.perf_counter() - t0
    g = oracle.geom(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad)
    rng = np.random.default_rng(0)
    T = {0: layer.c * layer.r * layer.s, 1: layer.k * layer.r * layer.s, 2: layer.n * layer.p * layer.q}
    O = {0: layer.n * layer.k * layer.p * layer.q, 1: layer.n * layer.c * layer.h * layer.w,
         2: layer.k * layer.c * layer.r * layer.s}
    args = {0: (ox, ow, ex + ew), 1: (ody, ow, edy + ew), 2: (ox, ody, ex + edy)}

    def run(budget):
        # calibrate on a small sample, then size each direction to ~budget/3 seconds
        macs, secs, samples = 0, 0.0, {}
        for dirn in (0, 1, 2):
            m = max(16, 2_000_000 // T[dirn])
            idx = rng.choice(O[dirn], size=min(m, O[dirn]), replace=False)
            t0 = time.perf_counter()
            oracle.conv_at(g, dirn, args[dirn][0], args[dirn][1], args[dirn][2], L, idx, G)
            per = (time.perf_counter() - t0) / idx.size
            m2 = int(min(O[dirn], max(idx.size, (budget / 3.0) / max(per, 1e-9))))
            idx = rng.choice(O[dirn], size=m2, replace=False)
            t0 = time.perf_counter()
            oracle.conv_at(g, dirn, args[dirn][0], args[dirn][1], args[dirn][2], L, idx, G)
            secs += time.perf_counter() - t0
            macs += idx.size * T[dirn]
            samples[dirn] = int(idx.size)
        return 2.0 * macs / secs / 1e12, macs, secs, samples

    all_v, macs, secs, samples = run(budget_s)
    omp.omp_set_num_threads(1)
    try:
        one_v, _, one_secs, _ = run(budget_s / 3.0)
    finally:
        omp.omp_set_num_threads(threads)
    return {
        "value": round(all_v, 6),
        "unit": "TOPS",
        "cores": threads,
        "kind": "oracle",
        "cpu": _cpu_model(),
        "single_thread_value": round(one_v, 7),
        "sample": "oracle conv at %d fwd / %d bwd-data / %d bwd-wt sampled outputs (%.3g MAC, %.1f s on %d "
                  "threads; single thread %.1f s) of the same layer and chunk length; full quantisation of x, w, "
                  "dy %.2f s, not in value" % (samples[0], samples[1], samples[2], macs, secs, threads, one_secs, tq),
    }


LAYER_WORKLOADS = ("resnet50_conv4x_1x1", "vgg16_conv1_2_conv3_3", "resnet50_all_convs")
DIRECTIONS = (("fwd", "conv_fwd_"), ("bwd_data", "conv_bwd_data_"), ("bwd_wt", "conv_bwd_wt_"))


def layer_sweep(a, dev):
    """The whole step on every layer of the other benchmark workloads, each at
    its own size, rounding and seed (inputs from the same host recipe as the
    headline): step time, and per direction the convolution kernels' time per
    step (all launches of the direction, e.g. phases) with TOPS and the
    fraction of the peak of the product path that ran.  The network's first
    layer (3 input channels) is summed without its backward-data and DC(dx),
    which training does not use; its row still times them, in a second run of
    the full step."""
    from paper_1802_00930_amd.workloads import WORKLOADS, layer_inputs
    res = {}
    for name in LAYER_WORKLOADS:
        wl = WORKLOADS[name]
        rows, total_s, total_ops = [], 0.0, 0.0
        for i in range(len(wl.layers)):
            layer, x, w, dy = layer_inputs(wl, i)
            ops = 2.0 * layer.macs
            stem = name == "resnet50_all_convs" and layer.c == 3
            for rounding in wl.roundings:
                st = Step(layer, x, w, dy, a.chunk, rounding, wl.seed, a.path, dev, a.seg_chunks)
                sec, _ = timed(st, 3, 1)
                _, recs = timed(st, 3, 0, profile=True)
                full_sec = None
                if stem:  # the step training runs: no input gradient
                    full_sec = sec
                    st.bwd_data = False
                    sec, _ = timed(st, 3, 1)
                row = {"layer": layer.name, "shape": "N%d C%d %dx%d K%d %dx%d s%d p%d" % (
                    layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad),
                    "rounding": rounding, "step_ms": round(sec * 1e3, 4), "step_tops": round(3 * ops / sec / 1e12, 2)}
                for dname, prefix in DIRECTIONS:
                    ks = [(n_, ms) for n_, ms in recs if n_.startswith(prefix)]
                    dsec = sum(ms for _, ms in ks) / 3 * 1e-3
                    mfma = all(n_.endswith(("_mfma", "_i32")) for n_, _ in ks)
                    tops = ops / dsec / 1e12 if dsec > 0 else 0.0
                    row[dname] = {"us": round(dsec * 1e6, 2), "tops": round(tops, 1),
                                  "frac": round(tops / (PEAK_INT16_BYTESPLIT_TOPS if mfma else PEAK_VALU_DOT2_TOPS), 4),
                                  "path": "mfma" if mfma else "valu"}
                if stem:
                    row["step_ms"] = round(sec * 1e3, 4)
                    row["step_tops"] = round(2 * ops / sec / 1e12, 2)
                    row["step_ms_with_bwd_data"] = round(full_sec * 1e3, 4)
                    row["bwd_data_not_in_sum"] = True
                rows.append(row)
                total_s += sec
                total_ops += (2 if stem else 3) * ops
                del st
            del x, w, dy
        res[name] = {"layers": rows, "sum_step_ms": round(total_s * 1e3, 3),
                     "tops_over_steps": round(total_ops / total_s / 1e12, 2)}
    return res


def cold_timed(step, steps, flush_bytes=512 << 20):
    """Median seconds of one step whose inputs were pushed out of the caches
    first: a write of flush_bytes (twice the 256 MB Infinity Cache) runs
    before every timed step, outside its HIP-event bracket."""
    torch = step.torch
    junk = torch.empty(flush_bytes // 4, dtype=torch.float32, device="cuda:0")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for s, e in ev:
        junk.fill_(1.0)
        s.record()
        step.run()
        e.record()
    torch.cuda.synchronize()
    del junk
    return float(np.median([s.elapsed_time(e) for s, e in ev])) * 1e-3


def emit_detail(name, payload, sink):
    """One detail block as its own JSON line (printed before the headline
    line, which stays last and short) and, with --detail-out, in a file."""
    line = json.dumps({"detail": name, **payload})
    print(line, flush=True)
    if sink is not None:
        sink.write(line + "\n")
        sink.flush()


def main():
    a = parse()
    if a.copy_probe:
        copy_probe(a.copy_probe)
        return
    if a.peaks:
        measure_peaks()
        return
    if a.gpus != 1:
        print("bench.py: the DFP convolution path measures one GPU (its kernels work on one GPU's share); "
              "--gpus %d is not supported" % a.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1802_00930_amd.workloads import WORKLOADS, layer_inputs
    from paper_1802_00930_amd import dfp
    dfp.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    sink = open(a.detail_out, "w") if a.detail_out else None
    wl = WORKLOADS[WORKLOAD]
    layer, x, w, dy = layer_inputs(wl, 0)
    rounding, seed = wl.roundings[0], wl.seed
    ops_per_dir = 2.0 * layer.macs

    step = Step(layer, x, w, dy, a.chunk, rounding, seed, a.path, dev, a.seg_chunks)
    sec, _ = timed(step, a.steps, a.warmup)              # the headline: no per-launch events
    cold_sec = cold_timed(step, max(5, a.steps // 2))    # the same step after a 512 MB cache flush
    _, recs = timed(step, a.steps, 1, profile=True)      # per-kernel durations (HIP events)
    per_kernel = {}
    for name, ms in recs:
        per_kernel.setdefault(name, []).append(ms)
    kstats = {k: {"launches_per_step": len(v) / a.steps, "avg_ms": float(np.mean(v)),
                  "total_ms_per_step": float(np.sum(v)) / a.steps} for k, v in per_kernel.items()}
    conv_kernels = {k: v for k, v in kstats.items() if k.startswith("conv_")}
    dominant = max(conv_kernels, key=lambda k: conv_kernels[k]["total_ms_per_step"])
    dk = kstats[dominant]
    mfma = "mfma" in dominant
    peak = PEAK_INT16_BYTESPLIT_TOPS if mfma else PEAK_VALU_DOT2_TOPS
    achieved = ops_per_dir / (dk["avg_ms"] * 1e-3) / 1e12
    traffic = measured_traffic(dominant)
    per_dir = {}
    for k, v in conv_kernels.items():
        per_dir[k] = {"avg_ms": round(v["avg_ms"], 5),
                      "tops": round(ops_per_dir / (v["avg_ms"] * 1e-3) / 1e12, 3),
                      "frac": round(ops_per_dir / (v["avg_ms"] * 1e-3) / 1e12 / peak, 4)}
    emit_detail("headline_kernels", {
        "workload": WORKLOAD, "per_direction": per_dir,
        "kernels": {k: {kk: round(vv, 5) for kk, vv in v.items()} for k, v in kstats.items()},
        "traffic_detail": traffic, "cold_ms_per_step": round(cold_sec * 1e3, 4)}, sink)

    if not a.no_sweep:
        sweep = {}
        for L in (8, 16, 32, 64):
            s2 = Step(layer, x, w, dy, L, rounding, seed, a.path, dev, max(1, a.seg_chunks * a.chunk // L))
            t2, _ = timed(s2, max(3, a.steps // 2), 2)
            sweep[str(L)] = {"ms_per_step": round(t2 * 1e3, 4), "tops": round(3 * ops_per_dir / t2 / 1e12, 3)}
            del s2
        emit_detail("chunk_sweep", {"workload": WORKLOAD, "by_chunk_len": sweep}, sink)

    # the DFP-32-output variant of the same step (reported beside the headline)
    if not a.no_dfp32:
        s32 = StepDfp32(layer, x, w, dy, a.chunk, rounding, seed, a.path, dev, a.seg_chunks)
        t32, _ = timed(s32, a.steps, a.warmup)
        _, recs32 = timed(s32, a.steps, 1, profile=True)
        emit_detail("dfp32_outputs", {
            "ms_per_step": round(t32 * 1e3, 4), "tops": round(3 * ops_per_dir / t32 / 1e12, 3),
            "chunk_len_fwd_bwd_data": s32.d32.chunk_len, "kernels": kernel_table(recs32, a.steps)}, sink)
        del s32

    # DFP16 GEMM: ResNet-50's FC layer step and one large product (reported beside the headline)
    if not a.no_gemm:
        fc = FcStep(64, 2048, 1000, a.chunk, rounding, seed, dev)
        tf, _ = timed(fc, a.steps, a.warmup)
        _, rf = timed(fc, a.steps, 1, profile=True)
        big = GemmStep(4096, 4096, 4096, a.chunk, dev)
        nb = max(3, a.steps // 2)
        tb, _ = timed(big, nb, 2)
        _, rb = timed(big, nb, 1, profile=True)
        kb = kernel_table(rb, nb)
        gemm_tops = 2.0 * big.macs / (kb["gemm"]["avg_ms"] * 1e-3) / 1e12
        bfc = BlockedFcStep(64, 2048, 1000, a.chunk, 128, rounding, seed, dev)
        tbf, _ = timed(bfc, a.steps, a.warmup)
        _, rbf = timed(bfc, a.steps, 1, profile=True)
        bbig = BlockedGemmStep(4096, 4096, 4096, a.chunk, 128, dev)
        tbb, _ = timed(bbig, nb, 2)
        _, rbb = timed(bbig, nb, 1, profile=True)
        kbb = kernel_table(rbb, nb)
        bg_tops = 2.0 * bbig.macs / (kbb["gemm_blocked"]["avg_ms"] * 1e-3) / 1e12
        emit_detail("gemm", {
            "fc_2048x1000_b64": {"ms_per_step": round(tf * 1e3, 4), "tops": round(3 * 2.0 * fc.macs / tf / 1e12, 3),
                                 "kernels": kernel_table(rf, a.steps)},
            "gemm_4096x4096x4096": {"ms_per_call": round(tb * 1e3, 4),
                                    "tops_call": round(2.0 * big.macs / tb / 1e12, 3),
                                    "kernel_tops": round(gemm_tops, 3),
                                    "kernel_frac": round(gemm_tops / PEAK_INT16_BYTESPLIT_TOPS, 4), "kernels": kb},
            "blocked_fc_forward_bk128": {"ms_per_step": round(tbf * 1e3, 4), "kernels": kernel_table(rbf, a.steps)},
            "blocked_gemm_4096x4096x4096_bk128": {
                "ms_per_call": round(tbb * 1e3, 4), "kernel_tops": round(bg_tops, 3),
                "kernel_frac": round(bg_tops / PEAK_INT16_BYTESPLIT_TOPS, 4), "kernels": kbb}}, sink)
        del fc, big, bfc, bbig

    # BN + ReLU forward / backward on the conv output and SGD + Q_w on the weights
    if not a.no_train_ops:
        tr = TrainOpsStep(layer, rounding, seed, dev)
        ttr, _ = timed(tr, a.steps, a.warmup)
        _, rtr = timed(tr, a.steps, 1, profile=True)
        # algorithmic bytes per element: BN forward reads y twice and writes zq (6 B); backward reads y and dz
        # in each of its three passes and writes dyq (14 B); SGD reads w, v, dw and writes w, v, then the
        # quantiser reads w and writes wq (26 B)
        emit_detail("train_ops", {
            "ms_per_step": round(ttr * 1e3, 4), "bn_elems": tr.elems, "sgd_weights": tr.nw,
            "algorithmic_bytes": {"bn_relu_fwd": 6 * tr.elems, "bn_relu_bwd": 14 * tr.elems,
                                  "sgd_quantize": 26 * tr.nw},
            "hbm_gbs_whole_step": round((20 * tr.elems + 26 * tr.nw) / ttr / 1e9, 1),
            "kernels": kernel_table(rtr, a.steps)}, sink)
        del tr

    layer_sums = None
    if not a.no_layers:
        lay = layer_sweep(a, dev)
        layer_sums = {}
        for name, res in lay.items():
            emit_detail("layers", {"workload": name, **res}, sink)
            layer_sums[name] = {"sum_step_ms": res["sum_step_ms"], "tops": res["tops_over_steps"]}

    out = {
        "metric": METRIC,
        "value": round(3 * ops_per_dir / sec / 1e12, 4),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(sec * 1e3, 4),
        "cold_ms_per_step": round(cold_sec * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int16",
        "data": "synthetic",
        "config": {
            "workload": "ResNet-50 conv2_x 3x3 layer N=%d C=K=%d %dx%d s1 p1, DFP15, L=%d, G=%d, %s rounding seed %d; "
                        "step = Q(x)+Q(w)+Q(dy)+fwd+DC(y)+bwd-data+DC(dx)+bwd-wt"
                        % (layer.n, layer.c, layer.h, layer.w, a.chunk, a.seg_chunks, rounding, seed),
            "chunk_len": a.chunk, "seg_chunks": a.seg_chunks},
        "roofline": {
            "bound": "mfma" if mfma else "alu",
            "kernel": dominant,
            "achieved": round(achieved, 3),
            "peak": peak,
            "unit": "TOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": (traffic or {}).get("bytes"),
        },
    }
    if layer_sums is not None:
        out["layer_sums"] = layer_sums
    if not a.no_cpu:
        out["cpu_baseline"] = cpu_baseline(layer, x, w, dy, a.chunk, a.seg_chunks, rounding, seed, a.cpu_seconds)
    if sink is not None:
        sink.write(json.dumps(out) + "\n")
        sink.close()
    print(json.dumps(out, separators=(",", ":")), flush=True)


if __name__ == "__main__":
    main()

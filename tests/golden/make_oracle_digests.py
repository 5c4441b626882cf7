#!/usr/bin/env python3
"""Write SHA-256 digests of the CPU oracle's full outputs for every benchmark
workload (``oracle_digests.json`` beside this file).

For each layer, rounding mode and chunk length of a workload this runs the
oracle's whole chain on the seeded FP32 inputs of ``workloads.py``:

    Q(x), Q(w), Q(dy)                     (Sec. 3.1 Eq. 1-3)
    y  = fwd(x, w),    DC(y)              (Alg. 2, Sec. 4.3; Sec. 1 / 4.1)
    dx = bwd_data(dy, w), DC(dx)
    dw = bwd_wt(x, dy)                    (segments of G chunks)

and records, per tensor, the exponent and flags, the digest of all its bytes
and a 64-bit digest prefix of every 1 MiB tile (so that a mismatch can be
located), plus max |y| and max |dx| as FP32 bit patterns.  The GPU tests run
the same chain in the benchmark's launch configuration and compare digests.

Only the oracle and the input generators are called.  The full run is about
an hour of 8-core CPU time (ResNet-50's 53 layers at N = 64 dominate); the
file is rewritten after every case, and a case already present is skipped,
so an interrupted run resumes.

    python tests/golden/make_oracle_digests.py [--only WORKLOAD] [--threads N]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_digests.json")
TILE_BYTES = 1 << 20
SEG_CHUNKS_AT_64 = 16  # backward-weights segment size at L = 64, scaled as 16 * 64 / L for other L

# (workload, chunk lengths): every benchmark workload in the launch
# configuration the benchmark times
CASES = (
    ("layer16x32", (16,)),
    ("resnet50_conv2x_3x3", (64, 32, 16, 8)),
    ("resnet50_conv4x_1x1", (64,)),
    ("vgg16_conv1_2_conv3_3", (64,)),
    ("resnet50_all_convs", (64,)),
)


def seg_chunks(L: int) -> int:
    return max(1, SEG_CHUNKS_AT_64 * 64 // L)


def case_key(workload: str, index: int, rounding: str, L: int) -> str:
    return "%s/%d/%s/L%d" % (workload, index, rounding, L)


def digest(a: np.ndarray) -> dict:
    b = np.ascontiguousarray(a).reshape(-1).view(np.uint8)
    tiles = [hashlib.sha256(b[i:i + TILE_BYTES].tobytes()).hexdigest()[:16] for i in range(0, b.size, TILE_BYTES)]
    return {"sha256": hashlib.sha256(b.tobytes()).hexdigest(), "bytes": int(b.size), "tiles": tiles}


def amax_bits(y: np.ndarray) -> int:
    return int((y.reshape(-1).view(np.uint32) & np.uint32(0x7FFFFFFF)).max())


def run_case(oracle, wl, index, rounding, L):
    from paper_1802_00930_amd.workloads import layer_inputs
    layer, x, w, dy = layer_inputs(wl, index)
    rnd = oracle.ROUNDING[rounding]
    seed = wl.seed
    G = seg_chunks(L)
    rec = {"layer": layer.name, "shape": [layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s,
                                          layer.stride, layer.pad],
           "rounding": rounding, "L": L, "G": G, "seed": seed, "bits": 15}
    ox, ex, fx = oracle.quantize(x, 15, rnd, seed, oracle.ROLE_X)
    ow, ew, fw = oracle.quantize(w, 15, rnd, seed, oracle.ROLE_W)
    ody, edy, fdy = oracle.quantize(dy, 15, rnd, seed, oracle.ROLE_DY)
    del x, w, dy
    rec["q"] = {name: {"exp": int(e), "flags": int(f), **digest(q)}
                for name, q, e, f in (("x", ox, ex, fx), ("w", ow, ew, fw), ("dy", ody, edy, fdy))}
    g = oracle.geom(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad)
    rec["out"], rec["dc"] = {}, {}
    for name, direction, a, b, e, role in (("y", oracle.FWD, ox, ow, ex + ew, oracle.ROLE_Y),
                                           ("dx", oracle.BWD_DATA, ody, ow, edy + ew, oracle.ROLE_DX),
                                           ("dw", oracle.BWD_WT, ox, ody, ex + edy, None)):
        out, _, overflow = oracle.conv(g, direction, a, b, e, L, G)
        rec["out"][name] = {"overflow": int(overflow), "flags": int(oracle.output_flags(out)), **digest(out)}
        if role is not None:
            rec["out"][name]["amax_bits"] = amax_bits(out)
            qo, eo, fo = oracle.quantize(out, 15, rnd, seed, role)
            rec["dc"][name] = {"exp": int(eo), "flags": int(fo), **digest(qo)}
            del qo
        del out
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", default="", help="comma-separated workload names")
    ap.add_argument("--threads", type=int, default=0, help="oracle OpenMP threads (0: its default)")
    a = ap.parse_args()
    if a.threads:
        os.environ["OMP_NUM_THREADS"] = str(a.threads)
    sys.path.insert(0, ROOT)
    import oracle
    from paper_1802_00930_amd.workloads import WORKLOADS
    oracle.lib()
    db = {"generator": "tests/golden/make_oracle_digests.py", "tile_bytes": TILE_BYTES,
          "seg_chunks_at_64": SEG_CHUNKS_AT_64, "numpy": np.__version__, "cases": {}}
    if os.path.exists(OUT):
        db = json.load(open(OUT))
    only = set(filter(None, a.only.split(",")))
    for name, lens in CASES:
        if only and name not in only:
            continue
        wl = WORKLOADS[name]
        for L in lens:
            for rounding in wl.roundings:
                for i in range(len(wl.layers)):
                    key = case_key(name, i, rounding, L)
                    if key in db["cases"]:
                        continue
                    t0 = time.time()
                    db["cases"][key] = run_case(oracle, wl, i, rounding, L)
                    tmp = OUT + ".tmp"
                    with open(tmp, "w") as f:
                        json.dump(db, f, indent=0, sort_keys=True)
                    os.replace(tmp, OUT)
                    print("%-40s %7.1f s" % (key, time.time() - t0), flush=True)


if __name__ == "__main__":
    main()

"""GPU parity at the full sizes of every benchmark workload, in the launch
configuration the benchmark times (bench.Step: default path, the workload's
chunk length and rounding, backward-weights segments of G = 16 * 64 / L
chunks).

Every tensor of the chain is compared in full against the CPU oracle's own
chain: Q(x), Q(w), Q(dy) (INT16, exponent, flags), the three FP32
convolution outputs, the epilogue's max |y| / |dx|, and the down-converted
INT16 outputs with their exponents and flags.  The oracle side is stored as
SHA-256 digests (whole tensor and per 1 MiB tile) in
tests/golden/oracle_digests.json, written by make_oracle_digests.py, which
calls only the oracle and the seeded input generators; a mismatch names the
tiles that differ.  FP32 outputs must then be bit-identical (0 ulp, inside
the 1e-6 relative bound), INT16 tensors, exponents and flags equal.

INT32 chunk partials are compared on sampled 32 x 32 output tiles (a 32-row,
32-position block of the output) plus the first and last tile, evaluated one
by one by the oracle, from a second call that records them.
"""
import hashlib
import json
import os
import zlib

import numpy as np
import pytest
import torch

import bench
import oracle
from gpu_helpers import DEV, note, oracle_geom
from paper_1802_00930_amd import dfp
from paper_1802_00930_amd.workloads import WORKLOADS, layer_inputs

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "oracle_digests.json")
DB = json.load(open(GOLDEN)) if os.path.exists(GOLDEN) else {"cases": {}, "tile_bytes": 1 << 20}
TILE = DB["tile_bytes"]


def _digest(a: np.ndarray):
    b = np.ascontiguousarray(a).reshape(-1).view(np.uint8)
    tiles = [hashlib.sha256(b[i:i + TILE].tobytes()).hexdigest()[:16] for i in range(0, b.size, TILE)]
    return hashlib.sha256(b.tobytes()).hexdigest(), tiles


def _check(name, got: np.ndarray, ref: dict, problems: list):
    sha, tiles = _digest(got)
    if sha != ref["sha256"]:
        bad = [i for i, (g, r) in enumerate(zip(tiles, ref["tiles"])) if g != r]
        problems.append("%s: %d of %d 1 MiB tiles differ, first %s" % (name, len(bad), len(ref["tiles"]), bad[:8]))


def _tiles(rng, rows, cols, count):
    """Flat output indices of `count` sampled 32 x 32 tiles plus the first and
    the last tile of an output viewed as [rows][cols] (each tile: 32
    consecutive rows x 32 consecutive columns, clipped at the edges)."""
    nr, nc = (rows + 31) // 32, (cols + 31) // 32
    picks = {(0, 0), (nr - 1, nc - 1)}
    while len(picks) < min(count + 2, nr * nc):
        picks.add((int(rng.integers(0, nr)), int(rng.integers(0, nc))))
    idx = []
    for tr, tc in sorted(picks):
        r = np.arange(tr * 32, min(rows, tr * 32 + 32))
        c = np.arange(tc * 32, min(cols, tc * 32 + 32))
        idx.append((r[:, None] * cols + c[None, :]).reshape(-1))
    return np.unique(np.concatenate(idx)).astype(np.int64)


def _partial_tiles(step, direction, a, sa, b, sb, oa, ob, e, L, G, ntiles, seed):
    """Chunk partials of sampled output tiles, GPU (partials call) vs oracle."""
    layer = step.layer
    d = step.d
    g = oracle.geom(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad)
    rng = np.random.default_rng(seed)
    if direction == dfp.FWD:  # y [N][K][PQ]: rows (n, k), columns pixels
        rows, cols = layer.n * layer.k, layer.p * layer.q
        out_shape = (layer.n, layer.k, layer.p, layer.q)
    elif direction == dfp.BWD_DATA:  # dx [N][C][HW]
        rows, cols = layer.n * layer.c, layer.h * layer.w
        out_shape = (layer.n, layer.c, layer.h, layer.w)
    else:  # dw [K][CRS]
        rows, cols = layer.k, layer.c * layer.r * layer.s
        out_shape = (layer.k, layer.c, layer.r, layer.s)
    idx = _tiles(rng, rows, cols, ntiles)
    J = dfp.num_chunks(d, direction)
    O = int(np.prod(out_shape))
    out = torch.empty(out_shape, dtype=torch.float32, device=DEV)
    parts = torch.full((J, O), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
    ws = dfp.alloc_workspace(d, direction, DEV)
    if direction == dfp.FWD:
        dfp.dfp_conv_fwd(d, a, sa, b, sb, out, None, ws, parts)
    elif direction == dfp.BWD_DATA:
        dfp.dfp_conv_bwd_data(d, a, sa, b, sb, out, None, ws, parts)
    else:
        dfp.dfp_conv_bwd_weights(d, a, sa, b, sb, out, ws, parts)
    gp = parts[:, torch.from_numpy(idx).to(DEV)].cpu().numpy().T
    del parts, out, ws
    _, rp, _ = oracle.conv_at(g, direction, oa, ob, e, L, idx, G, want_partials=True)
    bad = np.nonzero((gp != rp).any(axis=1))[0]
    assert bad.size == 0, "dir %d: partials differ at %d of %d sampled outputs, first flat index %d" % (
        direction, bad.size, idx.size, idx[bad[0]])


# partial-tile budget per workload (tiles per direction; backward-weights
# outputs each reduce over N*P*Q products, so fewer of them)
PARTIAL_TILES = {"layer16x32": (64, 64, 64), "resnet50_conv2x_3x3": (64, 64, 64), "resnet50_conv4x_1x1": (64, 64, 64),
                 "vgg16_conv1_2_conv3_3": (64, 64, 4), "resnet50_all_convs": (16, 16, 4)}


@pytest.mark.parametrize("key", sorted(DB["cases"]))
def test_full_chain_against_oracle_digests(key):
    case = DB["cases"][key]
    wname, index, rounding, _ = key.split("/")
    wl = WORKLOADS[wname]
    layer, x, w, dy = layer_inputs(wl, int(index))
    L, G, seed = case["L"], case["G"], case["seed"]
    assert list(case["shape"]) == [layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride,
                                   layer.pad] and case["bits"] == 15
    note("full chain %s (L=%d, G=%d)" % (key, L, G))
    step = bench.Step(layer, x, w, dy, L, rounding, seed, dfp.PATH_AUTO, DEV, G)
    assert step.d.seg_chunks == G
    step.run()
    torch.cuda.synchronize()
    problems = []
    for name, q, sc in (("x", step.qx, step.sx), ("w", step.qw, step.sw), ("dy", step.qdy, step.sdy)):
        s = dfp.read_scale(sc)
        ref = case["q"][name]
        if (s["exp"], s["flags"]) != (ref["exp"], ref["flags"]):
            problems.append("Q(%s): exp/flags %s vs oracle %s" % (name, (s["exp"], s["flags"]), (ref["exp"], ref["flags"])))
        _check("Q(%s)" % name, q.cpu().numpy(), ref, problems)
    for name, t in (("y", step.y), ("dx", step.dx), ("dw", step.dw)):
        _check(name, t.cpu().numpy(), case["out"][name], problems)
    for name, sc, q in (("y", step.sy, step.qy), ("dx", step.sdx, step.qdx)):
        s = dfp.read_scale(sc)
        ref = case["dc"][name]
        if s["amax_bits"] != case["out"][name]["amax_bits"]:
            problems.append("max|%s| bits %#x vs oracle %#x" % (name, s["amax_bits"], case["out"][name]["amax_bits"]))
        if (s["exp"], s["flags"]) != (ref["exp"], ref["flags"]):
            problems.append("DC(%s): exp/flags %s vs oracle %s" % (name, (s["exp"], s["flags"]), (ref["exp"], ref["flags"])))
        _check("DC(%s)" % name, q.cpu().numpy(), ref, problems)
    assert not problems, "%s:\n  %s" % (key, "\n  ".join(problems))

    # INT32 chunk partials on sampled output tiles (operands are the oracle's, equal to the GPU's by now)
    rnd = oracle.ROUNDING[rounding]
    ox, ex, _ = oracle.quantize(x, 15, rnd, seed, oracle.ROLE_X)
    ow, ew, _ = oracle.quantize(w, 15, rnd, seed, oracle.ROLE_W)
    ody, edy, _ = oracle.quantize(dy, 15, rnd, seed, oracle.ROLE_DY)
    nt = PARTIAL_TILES[wname]
    s0 = zlib.crc32(key.encode())
    for direction, a, sa, b, sb, oa, ob, e in (
            (dfp.FWD, step.qx, step.sx, step.qw, step.sw, ox, ow, ex + ew),
            (dfp.BWD_DATA, step.qdy, step.sdy, step.qw, step.sw, ody, ow, edy + ew),
            (dfp.BWD_WT, step.qx, step.sx, step.qdy, step.sdy, ox, ody, ex + edy)):
        note("  partials dir %d" % direction)
        _partial_tiles(step, direction, a, sa, b, sb, oa, ob, e, L, G, nt[direction], s0 + direction)
    del step
    torch.cuda.empty_cache()


def test_digest_file_covers_every_benchmark_workload():
    """Every layer, rounding and chunk length of the benchmark workloads has
    its oracle digests."""
    need = []
    for name, lens in (("layer16x32", (16,)), ("resnet50_conv2x_3x3", (64, 32, 16, 8)), ("resnet50_conv4x_1x1", (64,)),
                       ("vgg16_conv1_2_conv3_3", (64,)), ("resnet50_all_convs", (64,))):
        wl = WORKLOADS[name]
        for L in lens:
            for r in wl.roundings:
                for i in range(len(wl.layers)):
                    need.append("%s/%d/%s/L%d" % (name, i, r, L))
    missing = [k for k in need if k not in DB["cases"]]
    assert not missing, "%d cases without oracle digests, e.g. %s" % (len(missing), missing[:3])


def test_resnet50_conv2x_3x3_dfp32_full():
    """The benchmark layer through the single-chunk DFP-32 outputs (forward and
    backward-data at L = C*R*S = K*R*S = 576) and the integer down-convert
    with the epilogue's max, every element against the oracle."""
    from gpu_helpers import GpuLayer
    wl = WORKLOADS["resnet50_conv2x_3x3"]
    layer, x, w, dy = layer_inputs(wl, 0)
    L = layer.c * layer.r * layer.s
    gl = GpuLayer(layer.n, layer.c, layer.h, layer.w, layer.k, layer.r, layer.s, layer.stride, layer.pad, L=L,
                  rounding="stochastic", seed=wl.seed)
    g = oracle_geom(gl)
    rnd = oracle.ROUNDING["stochastic"]
    qx, sx = gl.quantize(x, dfp.ROLE_X)
    qw, sw = gl.quantize(w, dfp.ROLE_W)
    qdy, sdy = gl.quantize(dy, dfp.ROLE_DY)
    ox, ex, _ = oracle.quantize(x, 15, rnd, wl.seed, oracle.ROLE_X)
    ow, ew, _ = oracle.quantize(w, 15, rnd, wl.seed, oracle.ROLE_W)
    ody, edy, _ = oracle.quantize(dy, 15, rnd, wl.seed, oracle.ROLE_DY)
    torch.cuda.synchronize()
    assert np.array_equal(qx.cpu().numpy(), ox) and np.array_equal(qdy.cpu().numpy(), ody)
    assert np.array_equal(qw.cpu().numpy(), ow)
    for direction, a, sa, oa, ea, role, shape in ((dfp.FWD, qx, sx, ox, ex, dfp.ROLE_Y, gl.shape_y),
                                                  (dfp.BWD_DATA, qdy, sdy, ody, edy, dfp.ROLE_DX, gl.shape_x)):
        note("dfp32 layer %s dir %d" % (layer.name, direction))
        out = torch.empty(shape, dtype=torch.int32, device=DEV)
        so = dfp.new_scale(DEV)
        ws = dfp.alloc_workspace(gl.d, direction, DEV)
        f = dfp.dfp_conv_fwd_i32 if direction == dfp.FWD else dfp.dfp_conv_bwd_data_i32
        f(gl.d, a, sa, qw, sw, out, so, ws)
        q = torch.empty(shape, dtype=torch.int16, device=DEV)
        sq = dfp.new_scale(DEV)
        dfp.dfp_downconvert_i32(gl.d, role, out, so, q, sq, amax_ready=True)
        _, rparts, _ = oracle.conv(g, direction, oa, ow, ea + ew, L, 1, want_partials=True)
        rq, re, rf = oracle.downconvert_i32(rparts[0], ea + ew, 15, rnd, wl.seed, role)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().reshape(-1), rparts[0])
        assert np.array_equal(q.cpu().numpy().reshape(-1), rq)
        s = dfp.read_scale(sq)
        assert (s["exp"], s["flags"]) == (re, rf)
        del out, q, ws

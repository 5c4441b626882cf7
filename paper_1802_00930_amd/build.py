"""Build libdfp.so for gfx950 in-tree (hipcc, one object per HIP source)."""
from __future__ import annotations

import concurrent.futures as cf
import glob
import json
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdfp.so")
PEAKS_SRC = os.path.join(PKG, "peaks", "peaks.hip")
PEAKS_LIB = os.path.join(PKG, "libpeaks.so")
INCLUDE = os.path.join(os.path.dirname(PKG), "include")

ARCH = "gfx950"
# Packed FP32 VALU instructions are kept out of every kernel: hipcc would
# otherwise form them from ordinary float code.
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH, "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", INCLUDE,
]


def _hipcc():
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


# Kernels that wait for inline-assembly LDS reads in a later statement, per
# source: mangled-name fragment -> the macro that takes the kernel out of use
# when the built assembly fails asm_check (its launcher then runs a kernel
# whose LDS reads the compiler tracks or that waits inside the same asm).
SPLIT_READ_KERNELS = {
    "conv_bwdw_mfma.hip": {
        "k_bwdw_band_w8ILb0E": "DFP_ASM_UNSAFE_BAND_W8",
        "k_bwdw_band_w8ILb1E": "DFP_ASM_UNSAFE_BAND_W8_PARTIALS",
        "k_bwdw_band_skewILb0E": "DFP_ASM_UNSAFE_BAND_SKEW",
        "k_bwdw_band_skewILb1E": "DFP_ASM_UNSAFE_BAND_SKEW_PARTIALS",
        "k_bwdw_bandILb0E": "DFP_ASM_UNSAFE_BAND",
        "k_bwdw_bandILb1E": "DFP_ASM_UNSAFE_BAND_PARTIALS",
        "k_bwdw_flatILi": "DFP_ASM_UNSAFE_BAND_FLAT",
    },
    "conv_mfma.hip": {
        "k_conv_mfma_persistILb0ELb0E": "DFP_ASM_UNSAFE_PERSIST",
        "k_conv_mfma_persistILb1ELb0E": "DFP_ASM_UNSAFE_PERSIST_PARTIALS",
        "k_conv_mfma_persistILb0ELb1E": "DFP_ASM_UNSAFE_PERSIST_I32",
        "k_conv_mfma_skewILb0E": "DFP_ASM_UNSAFE_SKEW",
        "k_conv_mfma_skewILb1E": "DFP_ASM_UNSAFE_SKEW_PARTIALS",
    },
}
ASM_REPORT = os.path.join(BUILD, "asm_check.json")


def _compile(src: str, defines=()) -> str:
    name = os.path.basename(src)
    obj = os.path.join(BUILD, name + ".o")
    cmd = [_hipcc(), "-c", "-x", "hip", src, "-o", obj] + HIP_FLAGS + ["-D%s=1" % d for d in defines]
    if name in SPLIT_READ_KERNELS:
        cmd.append("-save-temps=obj")  # the device assembly of this very build, for asm_check
    res = subprocess.run(cmd, capture_output=True, text=True, cwd=BUILD)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, res.stdout, res.stderr))
    return obj


def _device_asm(src: str) -> str:
    stem = os.path.splitext(os.path.basename(src))[0]
    hits = glob.glob(os.path.join(BUILD, stem + "-hip-amdgcn-amd-amdhsa-" + ARCH + "*.s"))
    if len(hits) != 1:
        raise RuntimeError("device assembly of %s not found among the saved temporaries: %s" % (src, hits))
    return hits[0]


def _check_split_reads(src: str):
    """(kernels checked, macros of kernels that failed) for one source."""
    try:
        from . import asm_check
    except ImportError:  # run as a script
        import asm_check
    table = SPLIT_READ_KERNELS[os.path.basename(src)]
    report = asm_check.check_text(open(_device_asm(src)).read())
    bad = []
    for kernel, problems in report.items():
        if not problems:
            continue
        macro = [m for frag, m in table.items() if frag in kernel]
        if not macro:
            raise RuntimeError("asm_check: %s reads a register of an LDS read before its wait:\n  %s"
                               % (kernel, "\n  ".join(problems[:5])))
        bad.append(macro[0])
    return sorted(report), sorted(set(bad))


def build(verbose: bool = False) -> str:
    """Compile every csrc/*.hip for gfx950 and link libdfp.so.  Always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(sources))) as ex:
        objs = list(ex.map(_compile, sources))
    report = {}
    for i, src in enumerate(sources):
        name = os.path.basename(src)
        if name not in SPLIT_READ_KERNELS:
            continue
        kernels, bad = _check_split_reads(src)
        if bad:  # rebuild with the failing kernels out of use
            objs[i] = _compile(src, bad)
        missing = [f for f in SPLIT_READ_KERNELS[name] if not any(f in k for k in kernels)]
        if missing:
            raise RuntimeError("asm_check: kernels %s not found in the assembly of %s" % (missing, name))
        report[name] = {"kernels_checked": kernels, "out_of_use": bad}
    with open(ASM_REPORT, "w") as f:
        json.dump(report, f, indent=1)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (res.stdout, res.stderr))
    os.replace(tmp, LIB)
    build_peaks()
    if verbose:
        print("built", LIB, "and", PEAKS_LIB, file=sys.stderr)
    return LIB


def build_peaks() -> str:
    """The unit-ceiling microbenchmarks (bench.py --peaks); not part of libdfp."""
    tmp = PEAKS_LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), "-x", "hip", PEAKS_SRC, "-shared", "-o", tmp] + HIP_FLAGS
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (PEAKS_SRC, res.stdout, res.stderr))
    os.replace(tmp, PEAKS_LIB)
    return PEAKS_LIB


if __name__ == "__main__":
    build(verbose=True)

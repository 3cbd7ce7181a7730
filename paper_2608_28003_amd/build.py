"""Build ``libw8a8.so`` (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2608_28003_amd.build

Every translation unit is compiled with ``-ffp-contract=off`` (the quantisation
and epilogue arithmetic must stay one IEEE rounding per operation) and with
packed fp32 instructions disabled; no fast-math, no denormal flushing.
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "libw8a8.so")
ARCH = "gfx950"

CFLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: with AGPR accumulators the
    # 4-wave tile kernels copied every accumulator into AGPRs around each MFMA
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-result",
]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [_hipcc()] + CFLAGS + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, r.stdout, r.stderr))
    return obj


PEAK_LIB_PATH = os.path.join(HERE, "libw8a8_peak.so")


def _link(objs, path):
    tmp = path + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (r.stdout, r.stderr))
    # a shared library links with unresolved symbols; none of ours may be
    nm = subprocess.run(["nm", "-D", "-C", "--undefined-only", tmp], capture_output=True, text=True)
    missing = [l.split()[-1] for l in nm.stdout.splitlines() if "w8a8" in l]
    if nm.returncode == 0 and missing:
        os.remove(tmp)
        raise RuntimeError("unresolved library symbols: %s" % ", ".join(missing))
    os.replace(tmp, path)


def build(verbose: bool = True) -> str:
    """Compile every ``csrc/*.hip`` into ``libw8a8.so`` and ``csrc/peak/*.hip``
    (the benchmark's ceiling probes) into ``libw8a8_peak.so`` (always rebuilds)."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    peak_srcs = sorted(glob.glob(os.path.join(CSRC, "peak", "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs) + len(peak_srcs))) as ex:
        objs = list(ex.map(_compile, srcs + peak_srcs))
    _link(objs[:len(srcs)], LIB_PATH)
    _link(objs[len(srcs):], PEAK_LIB_PATH)
    if verbose:
        print("built", LIB_PATH, "and", PEAK_LIB_PATH, file=sys.stderr)
    return LIB_PATH


if __name__ == "__main__":
    build()

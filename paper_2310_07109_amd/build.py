"""Build libsc.so (the C-ABI library) for gfx950 with hipcc, in-tree.

    python -m paper_2310_07109_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libsc.so")
# the same library with SC_DEBUG: device-side argument checks and a synchronisation per call (include/sc.h)
DEBUG_OUT = os.path.join(HERE, "libsc_debug.so")
DEBUG_SOURCE = "sc_api.hip"  # the only source SC_DEBUG changes
# the VALU issue-rate probe behind the roofline figures (bench.py --probe-valu), a library of its own
PROBE_OUT = os.path.join(HERE, "libsc_probe.so")
PROBE_SOURCES = ["probe_valu.hip", "probe_lds.hip"]
BUILD_DIR = os.path.join(HERE, "_build")
SOURCES = ["sc_attention.hip", "sc_prune.hip", "sc_stack.hip", "sc_backward.hip", "sc_api.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    # Packed fp32 VALU forms are kept out of the code object.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in the unified VGPR file rather than in AGPRs: the
    # AGPR form copied every zero-initialised tile result in and out each tile
    # (v_accvgpr_write / read) and cost occupancy (the GEMM: 140 VGPRs + 64
    # AGPRs against 120 VGPRs).
    "-mllvm", "-amdgpu-mfma-vgpr-form",
]


def _compile(src: str, debug: bool = False) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ("_debug.o" if debug else ".o"))
    cmd = [HIPCC, *FLAGS, *(["-DSC_DEBUG"] if debug else []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return obj


def _link(objs: list, out: str) -> None:
    tmp = out + ".tmp"
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], capture_output=True,
                       text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES) + len(PROBE_SOURCES) + 1) as ex:
        objs = list(ex.map(_compile, SOURCES + PROBE_SOURCES))
        debug_obj = ex.submit(_compile, DEBUG_SOURCE, True).result()
    _link(objs[:len(SOURCES)], OUT)
    _link([debug_obj if s == DEBUG_SOURCE else o for s, o in zip(SOURCES, objs)], DEBUG_OUT)
    _link(objs[len(SOURCES):], PROBE_OUT)
    if verbose:
        print("built", OUT, DEBUG_OUT, "and", PROBE_OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

"""Build ``_lib/libscram.so`` (HIP, gfx950) from ``csrc/`` with hipcc.

Run as ``python -m paper_1905_10308_amd.build``; ``__graft_entry__.build()``
calls :func:`build`.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_DIR = os.path.join(HERE, "_lib")
LIB_PATH = os.path.join(LIB_DIR, "libscram.so")
# The same sources built with other launch settings: the lane-group kernels' tiles 16 wide and 4
# tall (not 8 x 8), every grid's tiles in bands of 3 tile columns (raster order below 65 tile
# columns), blocks in dispatch order (no XCD remap).  Every result the library documents as
# deterministic must come out bit-identical from both; the race checks load it beside the product.
ORDER_LIB_PATH = os.path.join(LIB_DIR, "libscram_order.so")
ORDER_DEFINES = ["-DSCRAM_LANE_TILE_SKEW=1", "-DSCRAM_BAND_TILES=3", "-DSCRAM_BAND_MAX=0", "-DSCRAM_XCD_REMAP=0"]
SOURCES = [os.path.join(CSRC, f) for f in ("scram_pm.hip", "scram_attend.hip", "scram_backward.hip", "scram_snis.hip",
                                             "scram_noalloc.hip", "scram_api.cpp")]
ARCH = "gfx950"

COMPILE_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # fixed operation order: explicit fmaf only, no implicit contraction
    "-ffp-contract=off",
    # never emit packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
LINK_FLAGS = [f"--offload-arch={ARCH}", "-shared", "-fPIC"]
# per-source additions: the attend step's matrix-core kernel keeps its accumulators in VGPRs (the
# compiler would otherwise copy them between AGPRs and VGPRs around every rescale)
EXTRA_FLAGS = {"scram_attend.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.isabs(cand) and os.path.exists(cand) or not os.path.isabs(cand)):
            return cand
    return "hipcc"


def _noise_free(res) -> list:
    # the host pass does not know the packed-fp32 feature and says so; drop that line
    return [ln for ln in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in ln and ln.strip()]


def build(verbose: bool = False) -> str:
    """Compile every source to an object (in parallel), then link the shared library; the same for
    the launch-order variant."""
    variants = [(LIB_PATH, "obj", []), (ORDER_LIB_PATH, "obj_order", ORDER_DEFINES)]
    jobs = []
    for _, sub, defines in variants:
        obj_dir = os.path.join(LIB_DIR, sub)
        os.makedirs(obj_dir, exist_ok=True)
        for src in SOURCES:
            obj = os.path.join(obj_dir, os.path.splitext(os.path.basename(src))[0] + ".o")
            cmd = [hipcc(), *COMPILE_FLAGS, *EXTRA_FLAGS.get(os.path.basename(src), []), *defines, f"-I{INCLUDE}",
                   f"-I{CSRC}", "-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            jobs.append((obj, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
    failed = []
    for obj, proc in jobs:
        out, err = proc.communicate()
        res = subprocess.CompletedProcess(proc.args, proc.returncode, out, err)
        if proc.returncode != 0:
            failed.append(f"{os.path.basename(obj)}:\n" + "\n".join(_noise_free(res)))
        elif verbose and _noise_free(res):
            print("\n".join(_noise_free(res)))
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
    for path, sub, _ in variants:
        objs = [os.path.join(LIB_DIR, sub, os.path.splitext(os.path.basename(src))[0] + ".o") for src in SOURCES]
        tmp = path + ".tmp"
        # -Bsymbolic: the library's own calls bind to its own definitions, also with the other
        # variant loaded in the same process
        cmd = [hipcc(), *LINK_FLAGS, "-Wl,-Bsymbolic", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("hipcc link failed:\n" + "\n".join(_noise_free(res)))
        os.replace(tmp, path)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

"""Build the HIP library libbsp.so for gfx950 (hipcc, in-tree).

    python -m paper_2111_11581_amd.build

Objects go to paper_2111_11581_amd/_build/, the shared library to
paper_2111_11581_amd/_build/libbsp.so.  Every HIP translation unit is compiled
with packed-fp32 instructions disabled (they are emitted by -O3 from plain
float code otherwise).
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "_build")
LIB = os.path.join(OUT, "libbsp.so")
ARCH = "gfx950"

SOURCES = ["bsp_pl_1.hip", "bsp_pl_2.hip", "bsp_pl_g.hip", "bsp_pw_b1.hip", "bsp_pw_b2.hip", "bsp_pw_f.hip", "bsp_fwd_b1_k1.hip", "bsp_fwd_b1_k24.hip", "bsp_fwd_b2.hip", "bsp_fwd_b3.hip", "bsp_fwd_b0.hip",
           "bsp_fwd_f.hip", "bsp_plan.cpp", "bsp_api.cpp", "bsp_prune.hip", "bsp_pack.hip",
           "bsp_conv.hip", "bsp_glue.hip", "bsp_stem.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def _compile(src: str) -> str:
    obj = os.path.join(OUT, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + COMMON + DEVICE + ["-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd.insert(1, "-xhip")
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libbsp.so.  Always rebuilds."""
    os.makedirs(OUT, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

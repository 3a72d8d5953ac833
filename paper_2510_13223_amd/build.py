"""Build libbana.so (HIP, gfx950 only) in-tree with hipcc.

    python -m paper_2510_13223_amd.build

Each source compiles to an object under ``_build/`` and the objects link into
``paper_2510_13223_amd/libbana.so``.  Packed-FP32 instructions are disabled for
all device code.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbana.so")
SOURCES = ["attn_partial.hip", "merge.hip", "migrate.hip", "validate.hip", "debug_rows.hip", "gather_read.hip",
           "scratch.hip",
           "bana_api.cpp"]

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def _compile(src: str, verbose: bool, build_dir: str, defines) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, *[f"-D{d}" for d in defines], "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


RACECHECK_LIB = os.path.join(PKG, "libbana_racecheck.so")


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile and link; ``out`` / ``defines`` allow side builds with other macros."""
    build_dir = BUILD if out == LIB else os.path.join(BUILD, os.path.basename(out) + ".objs")
    os.makedirs(build_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, build_dir, defines), SOURCES))
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)
    return out


def build_racecheck(verbose: bool = False) -> str:
    """The LDS race-check build (BANA_LDS_RACE_CHECK): delayed LDS writers and an extra barrier
    before every LDS read-back; a GPU test requires its results to equal the product build's."""
    return build(verbose, out=RACECHECK_LIB, defines=("BANA_LDS_RACE_CHECK",))


TIMELINE_LIB = os.path.join(PKG, "libbana_timeline.so")


def build_timeline(verbose: bool = False) -> str:
    """The wavefront-timeline build (BANA_WAVE_TIMELINE): every wavefront of the attention launches
    records clock readings (entry, schedule ready, first block, exit) for bana_debug_wave_timeline_read;
    a GPU test requires its results to equal the product build's."""
    return build(verbose, out=TIMELINE_LIB, defines=("BANA_WAVE_TIMELINE",))


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    print(build_racecheck(verbose="-v" in sys.argv))
    print(build_timeline(verbose="-v" in sys.argv))

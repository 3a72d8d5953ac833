"""Build the plain-C caller of the C ABI (tests/c/abi_roundtrip) with gcc.

It links libbana.so (the product library) and liboracle.so (the test oracle)
through run paths relative to the binary, so the tree can move.
"""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_roundtrip.c")
BIN = os.path.join(HERE, "abi_roundtrip")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    cmd = [
        "gcc", "-std=c11", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__",
        f"-I{os.path.join(ROOT, 'include')}", f"-I{os.path.join(ROCM, 'include')}", SRC, "-o", BIN + ".tmp",
        f"-L{os.path.join(ROOT, 'paper_2510_13223_amd')}", "-lbana", f"-L{os.path.join(ROOT, 'oracle')}", "-loracle",
        f"-L{os.path.join(ROCM, 'lib')}", "-lamdhip64", "-lm", "-fopenmp",
        "-Wl,-rpath,$ORIGIN/../../paper_2510_13223_amd:$ORIGIN/../../oracle",
    ]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed:\n{r.stderr}")
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())

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


# CPU builds with AddressSanitizer and UndefinedBehaviorSanitizer (host compilers only; no device
# code is built here).  Every sanitizer report is fatal.
SANITIZE = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{cmd[0]} failed:\n{r.stderr}")


def build_sanitized(out_dir: str) -> dict:
    """Sanitized CPU builds into out_dir:
    host        the library's host code (bana_api.cpp) with stub launchers, driven by a sweep
    oracle      the oracle (oracle.c), driven by a sweep of random small workloads
    host_lib    the library's host code with stub launchers as a shared library (for the ABI tests)
    oracle_lib  the oracle as a shared library (for the oracle pins)"""
    csrc = os.path.join(ROOT, "paper_2510_13223_amd", "csrc")
    inc = [f"-I{os.path.join(ROCM, 'include')}", f"-I{os.path.join(ROOT, 'include')}", f"-I{csrc}",
           "-D__HIP_PLATFORM_AMD__"]
    api = os.path.join(csrc, "bana_api.cpp")
    stubs = os.path.join(HERE, "sanitize_host.cpp")
    oracle_c = os.path.join(ROOT, "oracle", "oracle.c")
    out = {k: os.path.join(out_dir, v) for k, v in
           (("host", "sanitize_host"), ("oracle", "sanitize_oracle"), ("host_lib", "libbana_hostcheck.so"),
            ("oracle_lib", "liboracle_sanitized.so"))}
    _run(["g++", "-std=c++17", *SANITIZE, *inc, api, stubs, "-o", out["host"]])
    _run(["g++", "-std=c++17", *SANITIZE, "-fPIC", "-shared", "-DBANA_HOSTCHECK_LIBRARY", *inc, api, stubs, "-o",
          out["host_lib"]])
    _run(["gcc", "-std=c11", *SANITIZE, "-fopenmp", oracle_c, os.path.join(HERE, "sanitize_oracle.c"), "-o",
          out["oracle"], "-lm"])
    _run(["gcc", "-std=c11", *SANITIZE, "-fopenmp", "-fPIC", "-shared", oracle_c, "-o", out["oracle_lib"], "-lm"])
    return out


def sanitizer_preload() -> str:
    """LD_PRELOAD for a Python child that loads a sanitized shared library: the sanitizer runtimes
    first (they must come first), then whatever the environment already preloads."""
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True, check=True)
        libs.append(r.stdout.strip())
    rest = os.environ.get("LD_PRELOAD", "")
    return ":".join(libs + ([rest] if rest else []))


if __name__ == "__main__":
    print(build())

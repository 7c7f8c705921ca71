"""Compile tests/c_consumer/consumer.c, a plain C99 program that links
libgnnav.so and the HIP runtime's C API (no Python, no torch), into
tests/c_consumer/consumer.  Test infrastructure: __graft_entry__.build()
runs it after the library is built; tests run the binary.
Usage: python tests/c_consumer/build.py
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
BIN = os.path.join(HERE, "consumer")


def build(verbose: bool = True) -> str:
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        raise RuntimeError("no C compiler")
    lib_dir = os.path.join(ROOT, "paper_2404_09544_amd")
    if not os.path.exists(os.path.join(lib_dir, "libgnnav.so")):
        raise RuntimeError("build libgnnav.so first (paper_2404_09544_amd/build.py)")
    tmp = BIN + f".tmp{os.getpid()}"
    cmd = [cc, "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           os.path.join(HERE, "consumer.c"), "-o", tmp,
           "-L", lib_dir, "-lgnnav", "-Wl,-rpath,$ORIGIN/../../paper_2404_09544_amd",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, BIN)
    if verbose:
        print(f"[build] {BIN}", flush=True)
    return BIN


if __name__ == "__main__":
    build()
    sys.exit(0)

"""Build tests/c_abi/kq_abi_client (host-only C++ against the C ABI of
libkroquant.so and the C oracle) with hipcc.  Run by __graft_entry__.build()
after the library and the oracle are built; the GPU test only runs it."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "kq_abi_client.cpp")
BIN = os.path.join(HERE, "kq_abi_client")


def build() -> str:
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    # host code only (no kernels): gfx950 is named so that hipcc compiles no other target
    cmd = [hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17", "-Wall", SRC, "-I", os.path.join(ROOT, "include"),
           "-L", os.path.join(ROOT, "paper_2607_21446_amd"), "-l:libkroquant.so",
           "-L", os.path.join(ROOT, "oracle"), "-l:libkqoracle.so",
           "-Wl,-rpath,$ORIGIN/../../paper_2607_21446_amd:$ORIGIN/../../oracle", "-o", BIN + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())

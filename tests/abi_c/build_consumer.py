"""Compile the native ABI consumer (iabn_abi_check.cpp) against libiabn.so
and the oracle's C library; run by the build step, used by the GPU tests."""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "iabn_abi_check.cpp")
BIN = os.path.join(HERE, "iabn_abi_check")


def build() -> str:
    from paper_1712_02616_amd import build as hip_build

    cmd = [hip_build.hipcc(), "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           "-o", BIN + ".tmp", SRC,
           "-L", os.path.join(ROOT, "paper_1712_02616_amd"), "-liabn",
           "-L", os.path.join(ROOT, "oracle"), "-loracle_iabn",
           "-Wl,-rpath,$ORIGIN/../../paper_1712_02616_amd", "-Wl,-rpath,$ORIGIN/../../oracle"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("building the ABI consumer failed:\n%s\n%s" % (" ".join(cmd), res.stderr))
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())

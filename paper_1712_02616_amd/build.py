"""Compile libiabn.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

Each translation unit of ``csrc/`` compiles to an object file in parallel,
then one link makes the shared library.  ``build_probe`` compiles the
benchmark's bandwidth probes (``bench_probe.hip``) into a library of their
own, ``libiabn_probe.so``; libiabn does not contain or use them.
"""

from __future__ import annotations

import glob
import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
HEADERS = sorted(glob.glob(os.path.join(CSRC, "*.h"))) + [os.path.join(ROOT, "include", "iabn.h")]
LIB = os.path.join(HERE, "libiabn.so")
PROBE_SRC = os.path.join(HERE, "bench_probe.hip")
PROBE_LIB = os.path.join(HERE, "libiabn_probe.so")
ARCH = "gfx950"

FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         # Packed fp32 VALU instructions stay off on this target.
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; it is needed to build libiabn.so")


def _run(cmd):
    return subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)


def build(verbose: bool = False) -> str:
    """Always recompiles; writes libiabn.so next to this file atomically."""
    cc = hipcc()
    with tempfile.TemporaryDirectory(prefix="iabn_build_") as tmp:
        objs, procs = [], []
        for src in SOURCES:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            cmd = [cc] + FLAGS + ["-c", "-o", obj, src]
            objs.append(obj)
            procs.append((cmd, _run(cmd)))
        errors = []
        for cmd, p in procs:
            out, err = p.communicate()
            if p.returncode != 0:
                errors.append("%s\n%s" % (" ".join(cmd), err))
            elif verbose and err:
                print(err)
        if errors:
            raise RuntimeError("hipcc failed:\n" + "\n".join(errors))
        out = LIB + ".tmp%d" % os.getpid()
        cmd = [cc, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", out] + objs
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("link failed (%d):\n%s\n%s" % (res.returncode, " ".join(cmd), res.stderr))
        os.replace(out, LIB)
    return LIB


def build_probe() -> str:
    """Always recompiles libiabn_probe.so (the benchmark's bandwidth probes)."""
    out = PROBE_LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + FLAGS + ["-shared", "-o", out, PROBE_SRC]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s\n%s" % (res.returncode, " ".join(cmd), res.stderr))
    os.replace(out, PROBE_LIB)
    return PROBE_LIB


def is_built() -> bool:
    return os.path.exists(LIB)


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_probe())

"""The C ABI of libiabn on the host: exports, sizes, validation (CPU only).

Nothing here launches a kernel: every call made with placeholder pointers is
one that host-side validation must reject before touching the GPU.  These
tests are skipped where a GPU is visible, so that a validation bug can never
turn a placeholder pointer into a device access.
"""

import ctypes
import os
import re
import subprocess

import pytest
import torch

import paper_1712_02616_amd as iabn
from paper_1712_02616_amd import build as iabn_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "iabn.h")

OK, ERR_NULL, ERR_SHAPE, ERR_PARAM, ERR_DTYPE, ERR_WORKSPACE = 0, 1, 2, 3, 4, 5
F32, F16, BF16 = 0, 1, 2

no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                            reason="placeholder pointers are only safe without a GPU")


@pytest.fixture(scope="module")
def lib():
    return iabn.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(iabn_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("iabn_forward_train", "iabn_forward_eval", "iabn_backward",
                     "iabn_workspace_size", "iabn_status_string"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", iabn_build.LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (\w+)$", out, flags=re.M))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    for n in declared_functions():
        assert hasattr(lib, n)


def test_version_and_status_strings(lib):
    assert lib.iabn_version() >= 10000
    for code in range(7):
        assert lib.iabn_status_string(code).startswith(b"IABN_")
    assert b"unknown" in lib.iabn_status_string(99)


def _split(m, C):
    # The slicing rule documented in the library: about 512 blocks, at
    # least 4096 elements per slice, at most 1024 slices, slice length a
    # multiple of 8 elements.
    P = -(-512 // C)
    P = min(P, -(-m // 4096), 1024)
    P = max(P, 1)
    L = -(-m // P)
    L = -(-L // 8) * 8
    return -(-m // L)


@pytest.mark.parametrize("N,C,HW", [(2, 16, 64), (32, 256, 3136), (4, 256, 36864),
                                    (16, 2048, 784), (8, 256, 16384), (8, 512, 4096),
                                    (8, 1024, 4096), (8, 2048, 4096), (3, 5, 7), (1, 1, 2)])
def test_workspace_size(lib, N, C, HW):
    for dt in (F32, F16, BF16):
        assert lib.iabn_workspace_size(N, C, HW, dt) == C * _split(N * HW, C) * 4 * 32


def test_workspace_size_invalid(lib):
    assert lib.iabn_workspace_size(2, 3, 4, 7) == 0
    assert lib.iabn_workspace_size(-1, 3, 4, F32) == 0
    assert lib.iabn_workspace_size(2, 0, 4, F32) == 0
    assert lib.iabn_workspace_size(1 << 20, 4, 1 << 20, F32) == 0  # N*HW >= 2^31


FAKE = ctypes.c_void_p(0x1000)
NULL = ctypes.c_void_p(0)
STREAM = ctypes.c_void_p(0)


def fwd(lib, x=FAKE, dt=F32, ptrs=None, eps=1e-5, mom=0.1, slope=0.01, N=2, C=3, HW=4, ws=FAKE,
        wsb=1 << 20):
    ptrs = ptrs or [FAKE] * 6
    return lib.iabn_forward_train(x, dt, *ptrs, eps, mom, slope, N, C, HW, ws, wsb, STREAM)


@no_gpu
def test_forward_train_validation(lib):
    assert fwd(lib, dt=3) == ERR_DTYPE
    assert fwd(lib, N=-1) == ERR_SHAPE
    assert fwd(lib, N=1, HW=1) == ERR_SHAPE  # one value per channel: no variance
    assert fwd(lib, N=1 << 16, HW=1 << 16) == ERR_SHAPE
    assert fwd(lib, C=(1 << 20) + 1) == ERR_SHAPE
    assert fwd(lib, x=NULL) == ERR_NULL
    for k in range(6):
        ptrs = [FAKE] * 6
        ptrs[k] = NULL
        assert fwd(lib, ptrs=ptrs) == ERR_NULL
    assert fwd(lib, eps=0.0) == ERR_PARAM
    assert fwd(lib, eps=float("nan")) == ERR_PARAM
    assert fwd(lib, eps=float("inf")) == ERR_PARAM
    assert fwd(lib, slope=0.0) == ERR_PARAM
    assert fwd(lib, slope=-0.01) == ERR_PARAM
    assert fwd(lib, mom=-0.1) == ERR_PARAM
    assert fwd(lib, mom=1.5) == ERR_PARAM
    assert fwd(lib, mom=float("nan")) == ERR_PARAM
    assert fwd(lib, ws=NULL) == ERR_NULL
    assert fwd(lib, wsb=8) == ERR_WORKSPACE
    assert fwd(lib, ws=ctypes.c_void_p(0x1008)) == ERR_WORKSPACE
    assert fwd(lib, ws=ctypes.c_void_p(0x1004)) == ERR_WORKSPACE
    assert b"workspace" in lib.iabn_last_error()


@no_gpu
def test_empty_tensors_are_noops(lib):
    # C == 0: nothing to compute; no pointer is looked at.
    assert fwd(lib, x=NULL, ptrs=[NULL] * 6, C=0, ws=NULL, wsb=0) == OK
    assert lib.iabn_forward_eval(NULL, F16, NULL, NULL, NULL, NULL, 1e-5, 0.01, 4, 3, 0,
                                 STREAM) == OK
    assert lib.iabn_backward(NULL, NULL, BF16, NULL, NULL, NULL, NULL, NULL, 1e-5, 0.01, 2, 0, 5,
                             NULL, 0, STREAM) == OK


@no_gpu
def test_eval_validation(lib):
    def ev(x=FAKE, dt=F16, ptrs=None, eps=1e-5, slope=0.01, N=2, C=3, HW=4):
        ptrs = ptrs or [FAKE] * 4
        return lib.iabn_forward_eval(x, dt, *ptrs, eps, slope, N, C, HW, STREAM)
    assert ev(dt=-1) == ERR_DTYPE
    assert ev(C=-3) == ERR_SHAPE
    assert ev(x=NULL) == ERR_NULL
    for k in range(4):
        ptrs = [FAKE] * 4
        ptrs[k] = NULL
        assert ev(ptrs=ptrs) == ERR_NULL
    assert ev(eps=-1.0) == ERR_PARAM
    assert ev(slope=float("inf")) == ERR_PARAM


@no_gpu
def test_backward_validation(lib):
    def bw(z=FAKE, dz=FAKE, dt=BF16, ptrs=None, eps=1e-5, slope=0.01, N=2, C=3, HW=4, ws=FAKE,
           wsb=1 << 20):
        ptrs = ptrs or [FAKE] * 5
        return lib.iabn_backward(z, dz, dt, *ptrs, eps, slope, N, C, HW, ws, wsb, STREAM)
    assert bw(dt=5) == ERR_DTYPE
    assert bw(N=1, HW=1) == ERR_SHAPE
    assert bw(z=NULL) == ERR_NULL
    assert bw(dz=NULL) == ERR_NULL
    for k in range(5):
        ptrs = [FAKE] * 5
        ptrs[k] = NULL
        assert bw(ptrs=ptrs) == ERR_NULL
    assert bw(eps=0.0) == ERR_PARAM
    assert bw(slope=0.0) == ERR_PARAM
    assert bw(ws=NULL) == ERR_NULL
    assert bw(wsb=0) == ERR_WORKSPACE


@no_gpu
def test_phase_entry_points_validate(lib):
    assert lib.iabn_forward_stats(NULL, F32, 2, 3, 4, FAKE, 1 << 20, STREAM) == ERR_NULL
    assert lib.iabn_forward_stats(FAKE, F32, 2, 3, 4, FAKE, 0, STREAM) == ERR_WORKSPACE
    assert lib.iabn_forward_apply(FAKE, F32, *([FAKE] * 6), 1e-5, 2.0, 0.01, 2, 3, 4, FAKE,
                                  1 << 20, STREAM) == ERR_PARAM
    assert lib.iabn_backward_reduce(FAKE, FAKE, F16, FAKE, FAKE, -1.0, 2, 3, 4, FAKE, 1 << 20,
                                    STREAM) == ERR_PARAM
    assert lib.iabn_backward_apply(FAKE, FAKE, F16, FAKE, FAKE, FAKE, NULL, FAKE, 1e-5, 0.01, 2, 3,
                                   4, FAKE, 1 << 20, STREAM) == ERR_NULL


@no_gpu
def test_comparison_blocks_validate(lib):
    """The other blocks' entry points reject the same bad arguments, plus their
    extra tensors (z for the standard and checkpointing forwards, z and the
    saved mean for the standard backward) when NULL."""
    def sfwd(x=FAKE, z=FAKE, ptrs=None, mom=0.1, slope=0.01, N=2, C=3, HW=4, wsb=1 << 20):
        ptrs = ptrs or [FAKE] * 6
        return lib.iabn_std_forward_train(x, z, F16, *ptrs, 1e-5, mom, slope, N, C, HW, FAKE, wsb,
                                          STREAM)

    def cfwd(x=FAKE, z=FAKE, ptrs=None, mom=0.1, slope=0.01, N=2, C=3, HW=4, wsb=1 << 20):
        ptrs = ptrs or [FAKE] * 6
        return lib.iabn_ckpt_forward_train(x, z, BF16, *ptrs, 1e-5, mom, slope, N, C, HW, FAKE,
                                           wsb, STREAM)

    for f in (sfwd, cfwd):
        assert f(x=NULL) == ERR_NULL
        assert f(z=NULL) == ERR_NULL
        for k in range(6):
            ptrs = [FAKE] * 6
            ptrs[k] = NULL
            assert f(ptrs=ptrs) == ERR_NULL
        assert f(mom=2.0) == ERR_PARAM
        assert f(slope=-1.0) == ERR_PARAM
        assert f(N=1, HW=1) == ERR_SHAPE
        assert f(wsb=4) == ERR_WORKSPACE
        assert f(x=NULL, z=NULL, ptrs=[NULL] * 6, C=0) == OK

    def sbw(x=FAKE, z=FAKE, dz=FAKE, ptrs=None, eps=1e-5, wsb=1 << 20):
        ptrs = ptrs or [FAKE] * 6
        return lib.iabn_std_backward(x, z, dz, F32, *ptrs, eps, 0.01, 2, 3, 4, FAKE, wsb, STREAM)
    for kw in ("x", "z", "dz"):
        assert sbw(**{kw: NULL}) == ERR_NULL
    for k in range(6):
        ptrs = [FAKE] * 6
        ptrs[k] = NULL
        assert sbw(ptrs=ptrs) == ERR_NULL
    assert sbw(eps=0.0) == ERR_PARAM
    assert sbw(wsb=0) == ERR_WORKSPACE

    for fn in (lib.iabn_backward_ii, lib.iabn_ckpt_backward):
        assert fn(NULL, FAKE, F16, *([FAKE] * 5), 1e-5, 0.01, 2, 3, 4, FAKE, 1 << 20,
                  STREAM) == ERR_NULL
        assert fn(FAKE, FAKE, F16, *([FAKE] * 4), NULL, 1e-5, 0.01, 2, 3, 4, FAKE, 1 << 20,
                  STREAM) == ERR_NULL
        assert fn(FAKE, FAKE, F16, *([FAKE] * 5), 1e-5, 0.0, 2, 3, 4, FAKE, 1 << 20,
                  STREAM) == ERR_PARAM
        assert fn(FAKE, FAKE, 9, *([FAKE] * 5), 1e-5, 0.01, 2, 3, 4, FAKE, 1 << 20,
                  STREAM) == ERR_DTYPE

    assert lib.iabn_ckpt_recompute(NULL, FAKE, F32, FAKE, FAKE, 0.01, 2, 3, 4, STREAM) == ERR_NULL
    assert lib.iabn_ckpt_recompute(FAKE, FAKE, F32, FAKE, NULL, 0.01, 2, 3, 4, STREAM) == ERR_NULL
    assert lib.iabn_ckpt_recompute(FAKE, FAKE, F32, FAKE, FAKE, 0.0, 2, 3, 4, STREAM) == ERR_PARAM
    assert lib.iabn_ckpt_recompute(FAKE, FAKE, F32, FAKE, FAKE, 0.01, -2, 3, 4, STREAM) == ERR_SHAPE
    # one value per channel is fine without statistics
    assert lib.iabn_ckpt_recompute(NULL, NULL, F32, NULL, NULL, 0.01, 2, 0, 4, STREAM) == OK


def test_binding_rejects_bad_tensors():
    # Marshalling checks in the binding run before any library call.
    x = torch.zeros(2, 3, 4)
    g = torch.ones(3)
    with pytest.raises(ValueError):
        iabn.iabn_forward_train(x, g, g, g, g, g, g)  # CPU tensor
    with pytest.raises(ValueError):
        iabn.iabn_forward_eval(torch.zeros(2, 3, 4, dtype=torch.float64), g, g, g, g)


def test_divmagic_exhaustive_small_divisors(tmp_path):
    """The device index math divides by the row length with a multiply-high;
    check it against integer division on the CPU (same header)."""
    src = tmp_path / "t.c"
    src.write_text(r'''
#include <stdio.h>
#include <stdint.h>
#include "divmagic.h"
static uint64_t s = 88172645463325252ull;
static uint32_t rnd(void) { s ^= s << 13; s ^= s >> 7; s ^= s << 17; return (uint32_t)s; }
int main(void) {
  uint32_t ds[] = {1u, 2u, 3u, 7u, 49u, 98u, 196u, 392u, 784u, 3136u, 4096u, 9216u, 16384u,
                   36864u, 65535u, 65536u, 65537u, 1000003u, 2147483647u, 1073741825u};
  for (unsigned k = 0; k < sizeof ds / sizeof ds[0]; ++k) {
    iabn_divmagic_t m = iabn_divmagic_make(ds[k]);
    for (uint32_t n = 0; n < 200000u; ++n)
      if (iabn_divmagic_div(n, m) != n / ds[k]) { printf("FAIL d=%u n=%u\n", ds[k], n); return 1; }
    for (uint32_t n = 0x7fffffffu; n > 0x7fffffffu - 200000u; --n)
      if (iabn_divmagic_div(n, m) != n / ds[k]) { printf("FAIL d=%u n=%u\n", ds[k], n); return 1; }
  }
  for (int t = 0; t < 3000000; ++t) {
    uint32_t d = (rnd() & 0x7fffffffu) >> (rnd() % 31); if (!d) d = 1;
    uint32_t n = rnd() & 0x7fffffffu;
    iabn_divmagic_t m = iabn_divmagic_make(d);
    if (iabn_divmagic_div(n, m) != n / d) { printf("FAIL d=%u n=%u\n", d, n); return 1; }
  }
  for (uint32_t d = 1; d < 5000; ++d) {
    iabn_divmagic_t m = iabn_divmagic_make(d);
    for (uint32_t n = 0; n < 20000; n += 3)
      if (iabn_divmagic_div(n, m) != n / d) { printf("FAIL d=%u n=%u\n", d, n); return 1; }
  }
  printf("ok\n");
  return 0;
}
''')
    exe = tmp_path / "t"
    subprocess.run(["gcc", "-O2", "-I", os.path.join(ROOT, "paper_1712_02616_amd", "csrc"),
                    "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "ok", out.stdout

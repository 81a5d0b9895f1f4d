"""The C ABI from a native program: tests/abi_c/iabn_abi_check (built with
the library) allocates with hipMalloc, runs libiabn's training forward and
backward on a HIP stream of its own through include/iabn.h, and compares with
the oracle's C library (statistics, z and, for fp32 storage, the whole
chain; the per-channel identity sum dx = 0 for every storage type)."""

from __future__ import annotations

import os
import subprocess

import pytest
import torch

from gpu_helpers import say

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

HERE = os.path.dirname(os.path.abspath(__file__))
BIN = os.path.join(HERE, "abi_c", "iabn_abi_check")


@pytest.mark.parametrize("N,C,HW,dtype", [(2, 16, 64, 0), (4, 256, 1024, 1), (3, 300, 49, 2),
                                          (8, 512, 196, 0), (2, 1024, 4096, 1)])
def test_native_consumer(N, C, HW, dtype):
    assert os.path.exists(BIN), "build the ABI consumer first (__graft_entry__.build())"
    say("native ABI consumer N=%d C=%d HW=%d dtype=%d" % (N, C, HW, dtype))
    res = subprocess.run([BIN, str(N), str(C), str(HW), str(dtype), "7"], capture_output=True,
                         text=True, timeout=120)
    say(res.stdout.strip())
    assert res.returncode == 0, res.stdout + res.stderr

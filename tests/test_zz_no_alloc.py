"""iabn_forward_train_noalloc, the training forward for callers that cannot
allocate (its streaming kernels keep their partials in the library's static
scratch), through the C ABI against iabn_forward_train with a caller's
workspace: the same kernels, so the outputs must be bit-identical.  Two calls
in a row on shapes that take the streaming kernels (the ones that use the
scratch), the second smaller than the first, then a channel-resident shape
(no scratch), then the first shape again (the scratch holds the last call's
partials, which must not leak into the next call)."""

from __future__ import annotations

import ctypes

import pytest
import torch

import paper_1712_02616_amd as iabn
import workloads
from gpu_helpers import TORCH_DTYPES, GpuLayer, say

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

SHAPES = [
    # (N, C, HW, dtype, seed): streaming (C < 64), large then smaller
    (3, 32, 20008, "f16", 71),
    (2, 5, 1000, "f32", 72),
    # channel-resident (no scratch)
    (4, 256, 1024, "bf16", 73),
    # streaming with the most partials per call (C = 255 with big channels: 765 slices)
    (8, 255, 65536, "f16", 74),
    (3, 32, 20008, "f16", 71),
]


def run_noalloc(L: GpuLayer, eps, mom, slope):
    """iabn_forward_train_noalloc through the C ABI (raw pointers, the current stream)."""
    lib = iabn.load()
    N, C, HW = L.shape
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    code = iabn.DTYPE_CODES[L.x.dtype]
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = lib.iabn_forward_train_noalloc(p(L.x), code, p(L.gamma), p(L.beta), p(L.running_mean),
                                        p(L.running_var), p(L.save_mean), p(L.save_var), eps, mom,
                                        slope, N, C, HW, st)
    assert rc == 0, lib.iabn_last_error().decode()


def test_noalloc_equals_workspace_forward():
    eps, mom, slope = 1e-5, 0.1, 0.01
    for N, C, HW, dtype, seed in SHAPES:
        inp = workloads.make_layer(N, C, HW, dtype, seed, dz_std=0.1, gamma_sign=True)
        plan = iabn.iabn_plan("forward_train", TORCH_DTYPES[dtype], N, C, HW)
        say("noalloc forward %s shape=%s channel_resident=%d" % (dtype, (N, C, HW),
                                                                 plan["channel_resident"]))
        A = GpuLayer(inp)
        A.forward_train(eps, mom, slope)
        B = GpuLayer(inp)
        run_noalloc(B, eps, mom, slope)
        torch.cuda.synchronize()
        for k in ("x", "save_mean", "save_var", "running_mean", "running_var"):
            assert torch.equal(getattr(A, k), getattr(B, k)), (k, (N, C, HW, dtype))


def test_noalloc_validates_like_the_workspace_forward():
    inp = workloads.make_layer(2, 5, 1000, "f32", 75)
    L = GpuLayer(inp)
    before = L.x.clone()
    say("noalloc error paths")
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_forward_train_noalloc(L.x, L.gamma, L.beta, L.running_mean, L.running_var,
                                        L.save_mean, L.save_var, 1e-5, 0.1, 0.0)
    assert e.value.status == 3
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_forward_train_noalloc(L.x, L.gamma, L.beta, L.running_mean, L.running_var,
                                        L.save_mean, L.save_var, 1e-5, 1.5, 0.01)
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert torch.equal(L.x, before)

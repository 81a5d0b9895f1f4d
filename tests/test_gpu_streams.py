"""Calls on several HIP streams at once.

The library keeps no device state between calls: everything a call needs is
in its arguments (tensors, parameters, the workspace) and it enqueues only on
the stream it is given.  Two layers run concurrently on two streams (each
with its own workspace) give bit for bit what they give one after the other.
"""

from __future__ import annotations

import pytest
import torch

import paper_1712_02616_amd as iabn
import workloads
from gpu_helpers import TORCH_DTYPES, say, to_device

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]


def _layer(shape, dtype, seed):
    N, C, HW = shape
    inp = workloads.make_layer(N, C, HW, dtype, seed=seed, dz_std=0.1)
    dev = torch.device("cuda")
    L = dict(x0=to_device(inp.x, dtype), dz0=to_device(inp.dz, dtype),
             g=torch.from_numpy(inp.gamma).to(dev), b=torch.from_numpy(inp.beta).to(dev),
             ws=torch.empty(max(iabn.iabn_workspace_size(N, C, HW, TORCH_DTYPES[dtype]), 1),
                            dtype=torch.uint8, device=dev))
    for k in ("rm", "rv", "sm", "sv", "dg", "db"):
        L[k] = torch.empty(C, device=dev)
    return L


def _run(L, stream):
    with torch.cuda.stream(stream):
        L["x"] = L["x0"].clone()
        L["dz"] = L["dz0"].clone()
        L["rm"].fill_(0.0)
        L["rv"].fill_(1.0)
        for _ in range(3):  # repeated passes keep the two streams overlapping
            L["x"].copy_(L["x0"])
            L["dz"].copy_(L["dz0"])
            iabn.iabn_forward_train(L["x"], L["g"], L["b"], L["rm"], L["rv"], L["sm"], L["sv"],
                                    workspace=L["ws"], stream=stream)
            iabn.iabn_backward(L["x"], L["dz"], L["g"], L["b"], L["sv"], L["dg"], L["db"],
                               workspace=L["ws"], stream=stream)


def test_two_streams_match_sequential():
    layers = [_layer((8, 1024, 4096), "f16", 91), _layer((4, 24, 20008), "f32", 92)]
    say("streams: sequential")
    s0 = torch.cuda.current_stream()
    for L in layers:
        _run(L, s0)
    torch.cuda.synchronize()
    ref = [{k: L[k].clone() for k in ("x", "dz", "rm", "rv", "sm", "sv", "dg", "db")} for L in layers]
    say("streams: concurrent")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(s0)
    for L, s in zip(layers, streams):
        _run(L, s)
    for s in streams:
        s0.wait_stream(s)
    torch.cuda.synchronize()
    for L, r in zip(layers, ref):
        for k, v in r.items():
            assert torch.equal(L[k], v), k


def test_side_stream_library_workspace():
    """No workspace given and a stream that is not torch's current one: the
    workspace the binding allocates is released when the call returns, while
    the kernels still wait behind a long kernel on that stream; the current
    stream allocates and overwrites blocks of the same size meanwhile, and the
    results still match a plain run (the streaming kernels, which use the
    workspace)."""
    shape = (4, 24, 20008)
    L = _layer(shape, "f32", 93)
    nbytes = L["ws"].numel()
    s0 = torch.cuda.current_stream()

    def fresh():
        L["x"] = L["x0"].clone()
        L["dz"] = L["dz0"].clone()
        L["rm"].fill_(0.0)
        L["rv"].fill_(1.0)

    say("side stream: reference")
    fresh()
    iabn.iabn_forward_train(L["x"], L["g"], L["b"], L["rm"], L["rv"], L["sm"], L["sv"])
    iabn.iabn_backward(L["x"], L["dz"], L["g"], L["b"], L["sv"], L["dg"], L["db"])
    torch.cuda.synchronize()
    ref = {k: L[k].clone() for k in ("x", "dz", "rm", "rv", "sm", "sv", "dg", "db")}
    say("side stream: library workspace")
    side = torch.cuda.Stream()
    for _ in range(3):
        fresh()
        side.wait_stream(s0)
        with torch.cuda.stream(side):
            torch.cuda._sleep(2_000_000)  # keeps the side stream busy for a while
        iabn.iabn_forward_train(L["x"], L["g"], L["b"], L["rm"], L["rv"], L["sm"], L["sv"],
                                stream=side)
        junk = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        junk.fill_(0xFF)
        iabn.iabn_backward(L["x"], L["dz"], L["g"], L["b"], L["sv"], L["dg"], L["db"], stream=side)
        junk = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        junk.fill_(0x7F)
        s0.wait_stream(side)
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(L[k], v), k

"""Maximum sizes: tensors with more than 2^32 elements, the maximum channel
count, channels of hundreds of millions of values, through the C ABI against
the oracle on sampled channels (channels are independent, so a channel's
oracle result needs only that channel's data).

Inputs are drawn on the device with the seeded generator of ``workloads``
(too large to build on the host); the sampled channels' storage values are
copied to the host exactly and handed to the oracle.  As in the other parity
tests, the backward comparison gives both sides the same stored z: the
sampled channel of the GPU's z tensor is overwritten with the oracle's z
rounded to the storage type before the backward runs.
"""

from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_1712_02616_amd as iabn
import workloads
from gpu_helpers import TOL, TORCH_DTYPES, assert_close, max_rel, say, to_device

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

F32 = lambda v: float(np.float32(v))  # noqa: E731


@dataclasses.dataclass(frozen=True)
class Big:
    id: str
    N: int
    C: int
    HW: int
    dtype: str
    seed: int
    chans: tuple  # channels checked against the oracle


BIG = [
    # 4.8e9 elements per tensor: element offsets beyond 2^32 (channel 8 of
    # sample 1 starts at 17 * 2^28); 2^29 values per channel, streaming path.
    Big("over_2p32_elements_f16", 2, 9, 1 << 28, "f16", 41, (8,)),
    # The maximum channel count (2^20) with 16 values per channel: the
    # channel-resident path with 2-access channels, a 2^20-block grid.
    Big("max_channels_f32", 2, 1 << 20, 8, "f32", 42, (0, 1, 777, 65535, 524288, (1 << 20) - 1)),
    # One channel of 2^28 + 3 values with an odd row length: the one-element
    # path over a quarter billion values.
    Big("huge_odd_channel_bf16", 1, 1, (1 << 28) + 3, "bf16", 43, (0,)),
    # 256 channels of 2^20 values: the channel-resident path with most of each
    # channel read twice (8 of every 64 strips stay in registers).
    Big("huge_fused_channels_f16", 1, 256, 1 << 20, "f16", 44, (0, 255)),
]


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.to(torch.float64).cpu().numpy()


@pytest.mark.parametrize("case", BIG, ids=lambda c: c.id)
def test_max_size_parity(case):
    N, C, HW = case.N, case.C, case.HW
    say("large %s shape=%s: drawing inputs" % (case.id, (N, C, HW)))
    x, dz, prm = workloads.make_layer_device(N, C, HW, case.dtype, case.seed)
    chans = list(case.chans)
    x_s = host_f64(x[:, chans])
    dz_s = host_f64(dz[:, chans])
    gamma = torch.from_numpy(prm.gamma).cuda()
    beta = torch.from_numpy(prm.beta).cuda()
    rm = torch.zeros(C, device="cuda")
    rv = torch.ones(C, device="cuda")
    sm = torch.empty(C, device="cuda")
    sv = torch.empty(C, device="cuda")
    dg = torch.empty(C, device="cuda")
    db = torch.empty(C, device="cuda")
    ws = torch.empty(max(iabn.iabn_workspace_size(N, C, HW, TORCH_DTYPES[case.dtype]), 1),
                     dtype=torch.uint8, device="cuda")
    eps, mom, slope = 1e-5, 0.1, 0.01
    say("large %s: forward" % case.id)
    iabn.iabn_forward_train(x, gamma, beta, rm, rv, sm, sv, eps, mom, slope, workspace=ws)
    torch.cuda.synchronize()
    g_c, b_c = prm.gamma[chans], prm.beta[chans]
    say("large %s: oracle forward on channels %s" % (case.id, chans))
    fw = oracle.forward_train(x_s, g_c, b_c, prm.running_mean[chans], prm.running_var[chans],
                              F32(eps), F32(mom), F32(slope))
    assert_close("z", host_f64(x[:, chans]), fw["z"], case.dtype)
    for name, t in (("mean", sm), ("var", sv), ("running_mean", rm), ("running_var", rv)):
        assert max_rel(host_f64(t)[chans], fw[name]) <= TOL["f32"], name
    # Backward from the same stored z on both sides.
    z_store = workloads.f64_to_storage(fw["z"], case.dtype)
    x[:, chans] = to_device(z_store, case.dtype)
    var32 = fw["var"].astype(np.float32)
    sv[chans] = torch.from_numpy(var32).cuda()
    say("large %s: backward" % case.id)
    iabn.iabn_backward(x, dz, gamma, beta, sv, dg, db, eps, slope, workspace=ws)
    torch.cuda.synchronize()
    say("large %s: oracle backward" % case.id)
    bw = oracle.backward_i(workloads.storage_to_f64(z_store, case.dtype), dz_s, g_c, b_c, var32,
                           F32(eps), F32(slope))
    assert_close("dx", host_f64(dz[:, chans]), bw["dx"], case.dtype)
    assert max_rel(host_f64(dg)[chans], bw["dgamma"]) <= TOL[case.dtype], "dgamma"
    assert max_rel(host_f64(db)[chans], bw["dbeta"]) <= TOL[case.dtype], "dbeta"
    assert bool(torch.isfinite(dz).all()) and bool(torch.isfinite(x).all())

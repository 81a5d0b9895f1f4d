"""GPU parity over seeded random layer shapes: the library's own choices
(streaming or channel-resident kernels, ladder rung, strip or general
addressing, access width from the row length and the pointers' alignment)
exercised across shapes no hand-picked case names, each against the oracle
with the gates of the other parity tests: InPlace-ABN's forward and backward
(I and II), the standard block's and the proposed checkpointing's.

The shapes come from a fixed-seed generator, so every run tests the same
list; a shape that fails is reproduced by its id.  Tensors sit at an element
offset inside a larger buffer in about a third of the shapes (which breaks
16-byte alignment and takes narrower accesses), and the buffer around the
tensor is checked to be untouched.
"""

from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_1712_02616_amd as iabn
import workloads
from gpu_helpers import TORCH_DTYPES, TOL, assert_close, max_rel, say, to_device, to_f64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

F32 = lambda v: float(np.float32(v))  # noqa: E731
MAX_ELEMS = 3 << 20


@dataclasses.dataclass(frozen=True)
class Shape:
    id: str
    N: int
    C: int
    HW: int
    dtype: str
    offset: int  # elements before the tensor inside its buffer
    seed: int


def _shapes(count=48, seed=1712):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        dtype = ("f32", "f16", "bf16")[rng.integers(3)]
        C = int(rng.integers(1, 256)) if rng.random() < 0.35 else int(rng.integers(256, 1400))
        kind = rng.integers(4)
        if kind == 0:
            HW = int(rng.integers(1, 4000))
        elif kind == 1:
            HW = 8 * int(rng.integers(1, 600))
        elif kind == 2:
            HW = int((7, 14, 28, 56, 112)[rng.integers(5)]) ** 2
        else:
            HW = 1 << int(rng.integers(6, 15))
        N = int(rng.integers(1, 17))
        while N > 1 and N * C * HW > MAX_ELEMS:
            N = max(1, N // 2)
        while N * C * HW > MAX_ELEMS and C > 1:
            C = max(1, C // 2)
        if N * HW < 2:
            N = 2
        offset = int(rng.integers(1, 9)) if rng.random() < 0.35 else 0
        out.append(Shape("r%02d_%s_n%d_c%d_hw%d_o%d" % (i, dtype, N, C, HW, offset), N, C, HW, dtype,
                         offset, 5000 + i))
    return out


SHAPES = _shapes()
GUARD = 1024


def _placed(a: np.ndarray, dtype: str, offset: int, fill: float):
    """The storage values of `a` at `offset` inside a filled device buffer."""
    E = a.size
    buf = torch.full((offset + E + GUARD,), fill, dtype=TORCH_DTYPES[dtype], device="cuda")
    t = buf[offset: offset + E].view(a.shape)
    t.copy_(to_device(a, dtype))
    return buf, t


def _untouched(buf, offset, E, fill):
    return bool(torch.all(buf[:offset] == fill)) and bool(torch.all(buf[offset + E:] == fill))


@pytest.mark.parametrize("s", SHAPES, ids=lambda s: s.id)
def test_random_shape_parity(s):
    eps, mom, slope = 1e-5, 0.1, 0.01
    say("random %s" % s.id)
    inp = workloads.make_layer(s.N, s.C, s.HW, s.dtype, s.seed, dz_std=0.1, gamma_sign=True)
    E = s.N * s.C * s.HW
    xbuf, x = _placed(inp.x, s.dtype, s.offset, 5.5)
    gbuf, dz = _placed(inp.dz, s.dtype, s.offset, -2.25)
    dev = torch.device("cuda")
    gamma = torch.from_numpy(inp.gamma).to(dev)
    beta = torch.from_numpy(inp.beta).to(dev)
    rm = torch.from_numpy(inp.running_mean.copy()).to(dev)
    rv = torch.from_numpy(inp.running_var.copy()).to(dev)
    sm = torch.empty(s.C, device=dev)
    sv = torch.empty(s.C, device=dev)
    dg = torch.empty(s.C, device=dev)
    db = torch.empty(s.C, device=dev)

    # Forward against the oracle on the same x.
    iabn.iabn_forward_train(x, gamma, beta, rm, rv, sm, sv, eps, mom, slope)
    torch.cuda.synchronize()
    fw = oracle.forward_train(workloads.storage_to_f64(inp.x, s.dtype), inp.gamma, inp.beta,
                              inp.running_mean, inp.running_var, F32(eps), F32(mom), F32(slope))
    assert_close("z", to_f64(x), fw["z"], s.dtype)
    for name, t in (("mean", sm), ("var", sv), ("running_mean", rm), ("running_var", rv)):
        assert max_rel(to_f64(t), fw[name]) <= TOL["f32"], name

    # Backward against the oracle on the same stored z (the oracle's, rounded
    # to storage) and variance.
    z_store = workloads.f64_to_storage(fw["z"], s.dtype)
    x.copy_(to_device(z_store, s.dtype))
    var32 = fw["var"].astype(np.float32)
    sv.copy_(torch.from_numpy(var32).to(dev))
    iabn.iabn_backward(x, dz, gamma, beta, sv, dg, db, eps, slope)
    torch.cuda.synchronize()
    bw = oracle.backward_i(workloads.storage_to_f64(z_store, s.dtype),
                           workloads.storage_to_f64(inp.dz, s.dtype), inp.gamma, inp.beta, var32,
                           F32(eps), F32(slope))
    assert_close("dx", to_f64(dz), bw["dx"], s.dtype)
    assert max_rel(to_f64(dg), bw["dgamma"]) <= TOL[s.dtype], "dgamma"
    assert max_rel(to_f64(db), bw["dbeta"]) <= TOL[s.dtype], "dbeta"
    assert _untouched(xbuf, s.offset, E, 5.5) and _untouched(gbuf, s.offset, E, -2.25)


def _stored(s, inp, eps, mom, slope):
    fw = oracle.forward_train(workloads.storage_to_f64(inp.x, s.dtype), inp.gamma, inp.beta,
                              inp.running_mean, inp.running_var, F32(eps), F32(mom), F32(slope))
    return fw, workloads.f64_to_storage(fw["z"], s.dtype)


@pytest.mark.parametrize("s", SHAPES, ids=lambda s: s.id)
def test_random_shape_backward_ii(s):
    eps, mom, slope = 1e-5, 0.1, 0.01
    say("random II %s" % s.id)
    inp = workloads.make_layer(s.N, s.C, s.HW, s.dtype, s.seed, dz_std=0.1, gamma_sign=True)
    fw, z_store = _stored(s, inp, eps, mom, slope)
    E = s.N * s.C * s.HW
    zbuf, z = _placed(z_store, s.dtype, s.offset, 5.5)
    gbuf, dz = _placed(inp.dz, s.dtype, s.offset, -2.25)
    dev = torch.device("cuda")
    var32 = fw["var"].astype(np.float32)
    dg = torch.empty(s.C, device=dev)
    db = torch.empty(s.C, device=dev)
    iabn.iabn_backward_ii(z, dz, torch.from_numpy(inp.gamma).to(dev), torch.from_numpy(inp.beta).to(dev),
                          torch.from_numpy(var32).to(dev), dg, db, eps, slope)
    torch.cuda.synchronize()
    bw = oracle.backward_ii(workloads.storage_to_f64(z_store, s.dtype),
                            workloads.storage_to_f64(inp.dz, s.dtype), inp.gamma, inp.beta, var32,
                            F32(eps), F32(slope))
    assert_close("dx", to_f64(dz), bw["dx"], s.dtype)
    assert max_rel(to_f64(dg), bw["dgamma"]) <= TOL[s.dtype], "dgamma"
    assert max_rel(to_f64(db), bw["dbeta"]) <= TOL[s.dtype], "dbeta"
    assert _untouched(zbuf, s.offset, E, 5.5) and _untouched(gbuf, s.offset, E, -2.25)


@pytest.mark.parametrize("s", SHAPES, ids=lambda s: s.id)
def test_random_shape_standard_block(s):
    eps, mom, slope = 1e-5, 0.1, 0.01
    say("random standard %s" % s.id)
    inp = workloads.make_layer(s.N, s.C, s.HW, s.dtype, s.seed, dz_std=0.1, gamma_sign=True)
    fw, z_store = _stored(s, inp, eps, mom, slope)
    E = s.N * s.C * s.HW
    dev = torch.device("cuda")
    gamma = torch.from_numpy(inp.gamma).to(dev)
    beta = torch.from_numpy(inp.beta).to(dev)
    rm = torch.from_numpy(inp.running_mean.copy()).to(dev)
    rv = torch.from_numpy(inp.running_var.copy()).to(dev)
    sm = torch.empty(s.C, device=dev)
    sv = torch.empty(s.C, device=dev)
    xbuf, x = _placed(inp.x, s.dtype, s.offset, 5.5)
    zbuf, z = _placed(np.zeros_like(inp.x), s.dtype, s.offset, 1.75)
    iabn.iabn_std_forward_train(x, z, gamma, beta, rm, rv, sm, sv, eps, mom, slope)
    torch.cuda.synchronize()
    assert_close("z", to_f64(z), fw["z"], s.dtype)
    for name, t in (("mean", sm), ("var", sv), ("running_mean", rm), ("running_var", rv)):
        assert max_rel(to_f64(t), fw[name]) <= TOL["f32"], name
    assert torch.equal(x, to_device(inp.x, s.dtype)), "x must be kept"
    # Backward from x with the signs of the same stored z on both sides.
    z.copy_(to_device(z_store, s.dtype))
    mean32 = fw["mean"].astype(np.float32)
    var32 = fw["var"].astype(np.float32)
    gbuf, dz = _placed(inp.dz, s.dtype, s.offset, -2.25)
    dg = torch.empty(s.C, device=dev)
    db = torch.empty(s.C, device=dev)
    iabn.iabn_std_backward(x, z, dz, gamma, beta, torch.from_numpy(mean32).to(dev),
                           torch.from_numpy(var32).to(dev), dg, db, eps, slope)
    torch.cuda.synchronize()
    bw = oracle.backward_standard(workloads.storage_to_f64(inp.x, s.dtype),
                                  workloads.storage_to_f64(inp.dz, s.dtype), inp.gamma, inp.beta,
                                  mean32, var32, F32(eps), F32(slope),
                                  z=workloads.storage_to_f64(z_store, s.dtype))
    assert_close("dx", to_f64(dz), bw["dx"], s.dtype)
    assert max_rel(to_f64(dg), bw["dgamma"]) <= TOL[s.dtype], "dgamma"
    assert max_rel(to_f64(db), bw["dbeta"]) <= TOL[s.dtype], "dbeta"
    for buf, fill in ((xbuf, 5.5), (zbuf, 1.75), (gbuf, -2.25)):
        assert _untouched(buf, s.offset, E, fill)


@pytest.mark.parametrize("s", SHAPES, ids=lambda s: s.id)
def test_random_shape_checkpointing(s):
    """The proposed checkpointing: forward (x̂ over x, z out of place; z
    within the allowance of x̂'s storage rounding), recomputation equal to
    the forward's z, and the backward from the stored x̂."""
    from test_gpu_arms import assert_close_slack, ckpt_z_slack
    eps, mom, slope = 1e-5, 0.1, 0.01
    say("random checkpointing %s" % s.id)
    inp = workloads.make_layer(s.N, s.C, s.HW, s.dtype, s.seed, dz_std=0.1, gamma_sign=True)
    fw, _ = _stored(s, inp, eps, mom, slope)
    E = s.N * s.C * s.HW
    dev = torch.device("cuda")
    gamma = torch.from_numpy(inp.gamma).to(dev)
    beta = torch.from_numpy(inp.beta).to(dev)
    rm = torch.from_numpy(inp.running_mean.copy()).to(dev)
    rv = torch.from_numpy(inp.running_var.copy()).to(dev)
    sm = torch.empty(s.C, device=dev)
    sv = torch.empty(s.C, device=dev)
    xbuf, xh = _placed(inp.x, s.dtype, s.offset, 5.5)
    zbuf, z = _placed(np.zeros_like(inp.x), s.dtype, s.offset, 1.75)
    iabn.iabn_ckpt_forward_train(xh, z, gamma, beta, rm, rv, sm, sv, eps, mom, slope)
    torch.cuda.synchronize()
    xh_ref = oracle.normalize(workloads.storage_to_f64(inp.x, s.dtype), fw["mean"], fw["var"], F32(eps))
    assert_close("xhat", to_f64(xh), xh_ref, s.dtype)
    assert_close_slack("z", to_f64(z), fw["z"], s.dtype, ckpt_z_slack(xh_ref, inp.gamma, slope, s.dtype))
    for name, t in (("mean", sm), ("var", sv), ("running_mean", rm), ("running_var", rv)):
        assert max_rel(to_f64(t), fw[name]) <= TOL["f32"], name
    z2buf, z2 = _placed(np.zeros_like(inp.x), s.dtype, s.offset, 1.75)
    iabn.iabn_ckpt_recompute(xh, z2, gamma, beta, slope)
    torch.cuda.synchronize()
    assert torch.equal(z2, z)
    # Backward from the oracle's x̂ rounded to storage, on both sides.
    var32 = fw["var"].astype(np.float32)
    xh_store = workloads.f64_to_storage(xh_ref, s.dtype)
    xh.copy_(to_device(xh_store, s.dtype))
    gbuf, dz = _placed(inp.dz, s.dtype, s.offset, -2.25)
    dg = torch.empty(s.C, device=dev)
    db = torch.empty(s.C, device=dev)
    iabn.iabn_ckpt_backward(xh, dz, gamma, beta, torch.from_numpy(var32).to(dev), dg, db, eps, slope)
    torch.cuda.synchronize()
    dz64 = workloads.storage_to_f64(inp.dz, s.dtype)
    bw = oracle.backward_from_xhat(workloads.storage_to_f64(xh_store, s.dtype), dz64, inp.gamma,
                                   inp.beta, var32, F32(eps), F32(slope))
    A = np.abs(inp.gamma) / np.sqrt(var32.astype(np.float64) + F32(eps))
    assert_close("dx", to_f64(dz), bw["dx"], s.dtype, floor_abs=1e-3 * float(A.max() * np.abs(dz64).max()))
    assert max_rel(to_f64(dg), bw["dgamma"]) <= TOL[s.dtype], "dgamma"
    assert max_rel(to_f64(db), bw["dbeta"]) <= TOL[s.dtype], "dbeta"
    for buf, fill in ((xbuf, 5.5), (zbuf, 1.75), (z2buf, 1.75), (gbuf, -2.25)):
        assert _untouched(buf, s.offset, E, fill)

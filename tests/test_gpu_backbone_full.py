"""Whole-tensor parity of the benchmark's own layers: one full-size layer of
each of the four shape groups of the backbone sweep (fp16, N = 8:
(256, 128x128), (512, 64x64), (1024, 64x64), (2048, 64x64)), every channel
and every element compared with the oracle, through both ways into the
library (the fused entry points the benchmark times, and the phase entry
points).

Per layer and path:
  forward   z element by element at the fp16 gate; batch mean and variance
            and the running estimates at 1e-4 (fp32 arithmetic on exact
            storage values, whatever the storage type).
  backward  both sides start from the same stored z (the oracle's z rounded
            to fp16) and the same sigma^2; dx element by element, dgamma and
            dbeta per channel, at the fp16 gate and with no allowance; z is
            read-only.
  chain     GPU forward then GPU backward in place: against the oracle's
            backward on the GPU forward's own stored z and sigma^2 at the
            gate, and against the oracle's exact chain with the kink and
            storage-rounding allowances of ``chain_allowances``.

Channels are independent, so the oracle runs over chunks of channels (host
memory stays bounded); relative errors are floored at 1e-3 of the maximum
over the whole tensor, as in the other parity tests.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import TOL, GpuLayer, say, to_device, to_f64
from chain_allowance import check_same_inputs
from test_gpu_parity import F32, PATHS, chain_allowances, check_chain

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

W5 = workloads.WORKLOADS[5]
GROUPS = [0, 3, 7, 30]  # first layer of each (C, H=W) group
CHUNK_ELEMS = 1 << 23  # elements per oracle chunk


def chunks(N, C, HW):
    step = max(1, CHUNK_ELEMS // (N * HW))
    for c0 in range(0, C, step):
        yield c0, min(C, c0 + step)


def host_storage(t: torch.Tensor) -> np.ndarray:
    """Device fp16 tensor -> numpy float16 (exact)."""
    assert t.dtype == torch.float16
    return t.cpu().numpy()


def rel_err(got, ref, scale):
    """max |got - ref| / max(|ref|, 1e-3 * scale) with a given scale."""
    got = np.asarray(got, np.float64)
    assert np.all(np.isfinite(got)), "non-finite values"
    denom = np.maximum(np.abs(ref), 1e-3 * scale)
    denom = np.where(denom > 0, denom, 1.0)
    return float(np.max(np.abs(got - ref) / denom)) if ref.size else 0.0


def oracle_forward_chunked(inp, eps, momentum, slope):
    N, C, HW = inp.x.shape
    z = np.empty((N, C, HW))
    out = {k: np.empty(C) for k in ("mean", "var", "running_mean", "running_var")}
    for c0, c1 in chunks(N, C, HW):
        x = workloads.storage_to_f64(inp.x[:, c0:c1], W5.dtype)
        fw = oracle.forward_train(x, inp.gamma[c0:c1], inp.beta[c0:c1], inp.running_mean[c0:c1],
                                  inp.running_var[c0:c1], eps, momentum, slope)
        z[:, c0:c1] = fw["z"]
        for k in out:
            out[k][c0:c1] = fw[k]
    out["z"] = z
    return out


def oracle_backward_chunked(z, dz_store, gamma, beta, var, eps, slope):
    N, C, HW = z.shape
    dx = np.empty((N, C, HW))
    dg = np.empty(C)
    db = np.empty(C)
    for c0, c1 in chunks(N, C, HW):
        dz = workloads.storage_to_f64(dz_store[:, c0:c1], W5.dtype)
        bw = oracle.backward_i(z[:, c0:c1], dz, gamma[c0:c1], beta[c0:c1], var[c0:c1], eps, slope)
        dx[:, c0:c1] = bw["dx"]
        dg[c0:c1] = bw["dgamma"]
        db[c0:c1] = bw["dbeta"]
    return dict(dx=dx, dgamma=dg, dbeta=db)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("layer", GROUPS)
def test_backbone_layer_whole(layer, path):
    N, C, HW = W5.layers[layer]
    eps, mom, slope = F32(W5.eps), F32(W5.momentum), F32(W5.slope)
    tol = TOL[W5.dtype]
    say("backbone whole layer %d %s shape=%s: inputs" % (layer, path, (N, C, HW)))
    inp = workloads.workload_layer(W5, layer)

    # GPU forward, then the chain backward in place.
    say("backbone whole layer %d %s: GPU forward + backward" % (layer, path))
    L = GpuLayer(inp)
    L.forward_train(W5.eps, W5.momentum, W5.slope, path=path)
    torch.cuda.synchronize()
    z_gpu = host_storage(L.x)
    stats = {"mean": to_f64(L.save_mean), "var": to_f64(L.save_var),
             "running_mean": to_f64(L.running_mean), "running_var": to_f64(L.running_var)}
    L.backward(W5.eps, W5.slope, path=path)
    torch.cuda.synchronize()
    dx_chain = host_storage(L.dz)
    dg_chain, db_chain = to_f64(L.dgamma), to_f64(L.dbeta)

    # Forward against the oracle.
    say("backbone whole layer %d %s: oracle forward" % (layer, path))
    fw = oracle_forward_chunked(inp, eps, mom, slope)
    zscale = np.abs(fw["z"]).max()
    zerr = max(rel_err(z_gpu[:, c0:c1].astype(np.float64), fw["z"][:, c0:c1], zscale)
               for c0, c1 in chunks(N, C, HW))
    say("  z max rel err %.3e" % zerr)
    assert zerr <= tol, "z: %.3e > %.1e" % (zerr, tol)
    for k, got in stats.items():
        e = rel_err(got, fw[k], np.abs(fw[k]).max())
        say("  %s max rel err %.3e" % (k, e))
        assert e <= TOL["f32"], "%s: %.3e > %.1e" % (k, e, TOL["f32"])

    # Backward from the same stored z on both sides, no allowance.
    z_store = workloads.f64_to_storage(fw["z"], W5.dtype)
    var32 = fw["var"].astype(np.float32)
    say("backbone whole layer %d %s: GPU backward from the oracle's stored z" % (layer, path))
    z_dev = to_device(z_store, W5.dtype)
    L.dz.copy_(to_device(inp.dz, W5.dtype))
    L.backward(W5.eps, W5.slope, z=z_dev, save_var=torch.from_numpy(var32).cuda(), path=path)
    torch.cuda.synchronize()
    dx_strict = host_storage(L.dz)
    dg_strict, db_strict = to_f64(L.dgamma), to_f64(L.dbeta)
    assert torch.equal(z_dev, to_device(z_store, W5.dtype)), "the backward wrote z"
    del z_dev
    say("backbone whole layer %d %s: oracle backward (stored z)" % (layer, path))
    bw = oracle_backward_chunked(workloads.storage_to_f64(z_store, W5.dtype), inp.dz, inp.gamma,
                                 inp.beta, var32, eps, slope)
    dxscale = np.abs(bw["dx"]).max()
    dxerr = max(rel_err(dx_strict[:, c0:c1].astype(np.float64), bw["dx"][:, c0:c1], dxscale)
                for c0, c1 in chunks(N, C, HW))
    dgerr = rel_err(dg_strict, bw["dgamma"], np.abs(bw["dgamma"]).max())
    dberr = rel_err(db_strict, bw["dbeta"], np.abs(bw["dbeta"]).max())
    say("  dx %.3e dgamma %.3e dbeta %.3e" % (dxerr, dgerr, dberr))
    assert dxerr <= tol, "dx: %.3e > %.1e" % (dxerr, tol)
    assert dgerr <= tol, "dgamma: %.3e > %.1e" % (dgerr, tol)
    assert dberr <= tol, "dbeta: %.3e > %.1e" % (dberr, tol)
    del bw, z_store

    # The chain against the oracle's exact chain.
    say("backbone whole layer %d %s: oracle backward (exact chain)" % (layer, path))
    ref = oracle_backward_chunked(fw["z"], inp.dz, inp.gamma, inp.beta, fw["var"], eps, slope)
    scales = {k: np.abs(ref[k]).max() for k in ("dx", "dgamma", "dbeta")}
    ymax = np.abs(np.where(fw["z"] >= 0, fw["z"], fw["z"] / slope)).max()
    nflip = 0
    for c0, c1 in chunks(N, C, HW):
        zr = fw["z"][:, c0:c1]
        zg = z_gpu[:, c0:c1].astype(np.float64)
        flip = (zg >= 0) != (zr >= 0)
        if flip.any():
            y = np.where(zr >= 0, zr, zr / slope)
            assert np.all(np.abs(y[flip]) <= 2e-3 * ymax), "branch flips away from the kink"
            nflip += int(flip.sum())
        dz = workloads.storage_to_f64(inp.dz[:, c0:c1], W5.dtype)
        sub = {k: ref[k][c0:c1] if k != "dx" else ref["dx"][:, c0:c1] for k in ref}
        allow = chain_allowances(zr, dz, sub, fw["var"][c0:c1], inp.gamma[c0:c1],
                                 inp.beta[c0:c1], W5.eps, W5.slope, W5.dtype, flip)
        check_chain(dx_chain[:, c0:c1].astype(np.float64), dg_chain[c0:c1], db_chain[c0:c1], sub,
                    allow, flip, W5.dtype, scales=scales)
    say("  chain: %d kink flips of %d elements" % (nflip, N * C * HW))
    assert nflip <= max(8, 1e-5 * N * C * HW)
    del ref

    # The chain's backward against the oracle's on the GPU forward's own z and sigma^2.
    say("backbone whole layer %d %s: oracle backward (the GPU's stored z)" % (layer, path))
    same = oracle_backward_chunked(z_gpu.astype(np.float64), inp.dz, inp.gamma, inp.beta,
                                   stats["var"], eps, slope)
    scales = {k: np.abs(same[k]).max() for k in ("dx", "dgamma", "dbeta")}
    for c0, c1 in chunks(N, C, HW):
        sub = {k: same[k][c0:c1] if k != "dx" else same["dx"][:, c0:c1] for k in same}
        check_same_inputs(dx_chain[:, c0:c1].astype(np.float64), dg_chain[c0:c1], db_chain[c0:c1],
                          sub, W5.dtype, scales=scales)

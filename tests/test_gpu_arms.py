"""GPU parity of the other blocks of Sec. 3.2 against the oracle.

InPlace-ABN II (iabn_backward_ii), the standard block (iabn_std_forward_train,
iabn_std_backward: keeps x and z) and the proposed checkpointing
(iabn_ckpt_forward_train, iabn_ckpt_recompute, iabn_ckpt_backward: keeps
xhat), each through the C ABI, on the same seeded inputs as the InPlace-ABN
parity tests and with the same gates.  As there, the backward comparisons
hand both sides identical stored tensors (the oracle's outputs rounded to the
storage type), so both take the leaky-ReLU branch from the same values; the
chain comparisons run GPU forward then GPU backward against the oracle's
chain with the kink and storage-rounding allowances of the InPlace-ABN chain.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_1712_02616_amd as iabn
import workloads
from gpu_helpers import TORCH_DTYPES, TOL, assert_close, max_rel, say, to_device, to_f64
from chain_allowance import check_same_inputs
from test_gpu_parity import (ALL_CASES, CONFIG_CASES, EDGE_CASES, F32, STORE_U, Case,
                             chain_allowances, check_chain, make_inputs, oracle_forward)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

_BY_ID = {c.id: c for c in ALL_CASES}
# Streaming shapes (few channels, odd HW, ragged slices), every fused ladder
# rung and storage type, the two-channel blocks, and the numerically awkward
# cases.
ARM_CASES = [_BY_ID[k] for k in (
    "cfg1_tiny_f32", "cfg2_resnet_f32", "cfg3_segcrop_f16", "cfg4_wide_bf16", "odd_hw49_bf16",
    "hw1_f32", "n1_m2_f16", "ragged_slices_f16", "ragged_odd_f32", "all_negative_f16",
    "all_positive_bf16", "slope1_plain_bn_f32", "large_mean_f32", "eps_large_bf16",
    "manych_c600_f16", "manych_c520_f32", "manych_t256_c512_f16", "rung256x8_strip_f16",
    "rung256x8_strip_f32", "fewch_c128_f16", "fewch_c64_f32", "narrow8_hw196_f16",
    "narrow4_hw98_bf16", "narrow4_hw49_f32", "pair_c1536_f32", "pair_bwd_c512_f32",
    "triple_bwd_c768_f16")]
CHAIN_CASES = [_BY_ID[k] for k in ("cfg1_tiny_f32", "odd_hw49_f16", "ragged_slices_bf16",
                                   "manych_c520_f32", "manych_t256_c512_f16", "cfg4_wide_bf16")]


class Dev:
    """Per-channel tensors and workspace of one layer on the device."""

    def __init__(self, inp: workloads.LayerInputs):
        N, C, HW = inp.x.shape
        self.gamma = torch.from_numpy(inp.gamma).cuda()
        self.beta = torch.from_numpy(inp.beta).cuda()
        self.rm = torch.from_numpy(inp.running_mean.copy()).cuda()
        self.rv = torch.from_numpy(inp.running_var.copy()).cuda()
        self.mean = torch.empty(C, dtype=torch.float32, device="cuda")
        self.var = torch.empty(C, dtype=torch.float32, device="cuda")
        self.dgamma = torch.empty(C, dtype=torch.float32, device="cuda")
        self.dbeta = torch.empty(C, dtype=torch.float32, device="cuda")
        self.ws = torch.empty(max(iabn.iabn_workspace_size(N, C, HW, TORCH_DTYPES[inp.dtype]), 1),
                              dtype=torch.uint8, device="cuda")


def f64(a, dtype):
    return workloads.storage_to_f64(a, dtype)


def check_stats(D: Dev, ref):
    for k, t in (("mean", D.mean), ("var", D.var), ("running_mean", D.rm), ("running_var", D.rv)):
        assert max_rel(to_f64(t), ref[k]) <= TOL["f32"], k


def check_grads(D: Dev, dx, ref, dtype, scale=None):
    """``scale``: the natural size A*|dy| of dx's terms; it floors the relative
    error where dx cancels exactly (m = 2 with xhat stored as +-1: dx = 0)."""
    assert_close("dx", dx, ref["dx"], dtype, floor_abs=0.0 if scale is None else 1e-3 * scale)
    assert max_rel(to_f64(D.dgamma), ref["dgamma"]) <= TOL[dtype], "dgamma"
    assert max_rel(to_f64(D.dbeta), ref["dbeta"]) <= TOL[dtype], "dbeta"


def ckpt_z_slack(xh_ref, gamma, slope, dtype):
    """The checkpointing forward forms z from xhat as stored, so that the
    backward's recomputation reproduces it; its z differs from the exact one by
    f' |gamma| |xhat_stored - xhat| <= max(1, a) |gamma| u |xhat| (u: unit
    roundoff of the storage type plus a few fp32 roundings)."""
    return max(1.0, F32(slope)) * np.abs(np.asarray(gamma, np.float64))[None, :, None] * \
        STORE_U[dtype] * np.abs(xh_ref)


def ckpt_branch(xh_gpu, gamma, beta):
    """The branch the checkpointing kernels take: gamma*xhat + beta < 0 on the
    stored xhat (a product of two fp32-representable values is exact in
    double, so the one rounding of the sum keeps the sign, as the kernels'
    fused multiply-add does)."""
    g = np.asarray(gamma, np.float64)[None, :, None]
    b = np.asarray(beta, np.float64)[None, :, None]
    return g * xh_gpu + b < 0


def assert_close_slack(name, got, ref, dtype, slack):
    """assert_close with an absolute allowance per element."""
    got = np.asarray(got, np.float64)
    assert np.all(np.isfinite(got)), "%s has non-finite values" % name
    floor = np.maximum(np.abs(ref), 1e-3 * np.abs(ref).max())
    err = float(np.max(np.maximum(np.abs(got - ref) - slack, 0.0) / floor))
    assert err <= TOL[dtype], "%s: max rel err beyond allowance %.3e > %.1e (%s)" % (
        name, err, TOL[dtype], dtype)


def stored_backward_inputs(case: Case, inp):
    """The oracle's forward outputs rounded to what the library stores."""
    fw = oracle_forward(case, inp)
    z_store = workloads.f64_to_storage(fw["z"], case.dtype)
    mean32 = fw["mean"].astype(np.float32)
    var32 = fw["var"].astype(np.float32)
    return fw, z_store, mean32, var32


# ---------------------------------------------------------------- InPlace-ABN II


@pytest.mark.parametrize("case", ARM_CASES, ids=lambda c: c.id)
def test_backward_ii_parity(case):
    inp = make_inputs(case)
    fw, z_store, _, var32 = stored_backward_inputs(case, inp)
    say("backward II %s shape=%s" % (case.id, (case.N, case.C, case.HW)))
    D = Dev(inp)
    z = to_device(z_store, case.dtype)
    g = to_device(inp.dz, case.dtype)
    iabn.iabn_backward_ii(z, g, D.gamma, D.beta, torch.from_numpy(var32).cuda(), D.dgamma, D.dbeta,
                          case.eps, case.slope, workspace=D.ws)
    torch.cuda.synchronize()
    ref = oracle.backward_ii(f64(z_store, case.dtype), f64(inp.dz, case.dtype), inp.gamma, inp.beta,
                             var32, F32(case.eps), F32(case.slope))
    check_grads(D, to_f64(g), ref, case.dtype)
    assert torch.equal(z, to_device(z_store, case.dtype))


# ---------------------------------------------------------------- standard block


@pytest.mark.parametrize("case", ARM_CASES, ids=lambda c: c.id)
def test_std_forward_parity(case):
    inp = make_inputs(case)
    say("standard forward %s shape=%s" % (case.id, (case.N, case.C, case.HW)))
    D = Dev(inp)
    x = to_device(inp.x, case.dtype)
    z = torch.empty_like(x)
    iabn.iabn_std_forward_train(x, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, case.eps,
                                case.momentum, case.slope, workspace=D.ws)
    torch.cuda.synchronize()
    ref = oracle_forward(case, inp)
    assert_close("z", to_f64(z), ref["z"], case.dtype)
    check_stats(D, ref)
    assert torch.equal(x, to_device(inp.x, case.dtype)), "x must be kept"


@pytest.mark.parametrize("case", ARM_CASES, ids=lambda c: c.id)
def test_std_backward_parity(case):
    inp = make_inputs(case)
    fw, z_store, mean32, var32 = stored_backward_inputs(case, inp)
    say("standard backward %s shape=%s" % (case.id, (case.N, case.C, case.HW)))
    D = Dev(inp)
    x = to_device(inp.x, case.dtype)
    z = to_device(z_store, case.dtype)
    g = to_device(inp.dz, case.dtype)
    iabn.iabn_std_backward(x, z, g, D.gamma, D.beta, torch.from_numpy(mean32).cuda(),
                           torch.from_numpy(var32).cuda(), D.dgamma, D.dbeta, case.eps, case.slope,
                           workspace=D.ws)
    torch.cuda.synchronize()
    ref = oracle.backward_standard(f64(inp.x, case.dtype), f64(inp.dz, case.dtype), inp.gamma,
                                   inp.beta, mean32, var32, F32(case.eps), F32(case.slope),
                                   z=f64(z_store, case.dtype))
    check_grads(D, to_f64(g), ref, case.dtype)
    assert torch.equal(x, to_device(inp.x, case.dtype)) and torch.equal(z, to_device(z_store, case.dtype))


# ---------------------------------------------------------------- proposed checkpointing


@pytest.mark.parametrize("case", ARM_CASES, ids=lambda c: c.id)
def test_ckpt_forward_parity(case):
    inp = make_inputs(case)
    say("checkpointing forward %s shape=%s" % (case.id, (case.N, case.C, case.HW)))
    D = Dev(inp)
    xh = to_device(inp.x, case.dtype)
    z = torch.empty_like(xh)
    iabn.iabn_ckpt_forward_train(xh, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, case.eps,
                                 case.momentum, case.slope, workspace=D.ws)
    torch.cuda.synchronize()
    ref = oracle_forward(case, inp)
    xh_ref = oracle.normalize(f64(inp.x, case.dtype), ref["mean"], ref["var"], F32(case.eps))
    assert_close("xhat", to_f64(xh), xh_ref, case.dtype)
    assert_close_slack("z", to_f64(z), ref["z"], case.dtype,
                       ckpt_z_slack(xh_ref, inp.gamma, case.slope, case.dtype))
    check_stats(D, ref)
    # The backward's recomputation from the stored xhat gives back z exactly.
    z2 = torch.empty_like(z)
    iabn.iabn_ckpt_recompute(xh, z2, D.gamma, D.beta, case.slope)
    torch.cuda.synchronize()
    assert torch.equal(z2, z)


@pytest.mark.parametrize("case", ARM_CASES, ids=lambda c: c.id)
def test_ckpt_recompute_parity(case):
    inp = make_inputs(case)
    fw = oracle_forward(case, inp)
    xh_store = workloads.f64_to_storage(
        oracle.normalize(f64(inp.x, case.dtype), fw["mean"], fw["var"], F32(case.eps)), case.dtype)
    say("checkpointing recompute %s shape=%s" % (case.id, (case.N, case.C, case.HW)))
    D = Dev(inp)
    xh = to_device(xh_store, case.dtype)
    z = torch.empty_like(xh)
    iabn.iabn_ckpt_recompute(xh, z, D.gamma, D.beta, case.slope)
    torch.cuda.synchronize()
    ref = oracle.scale_shift_act(f64(xh_store, case.dtype), inp.gamma, inp.beta, F32(case.slope))
    assert_close("z", to_f64(z), ref, case.dtype)


@pytest.mark.parametrize("case", ARM_CASES, ids=lambda c: c.id)
def test_ckpt_backward_parity(case):
    inp = make_inputs(case)
    fw = oracle_forward(case, inp)
    var32 = fw["var"].astype(np.float32)
    xh_store = workloads.f64_to_storage(
        oracle.normalize(f64(inp.x, case.dtype), fw["mean"], fw["var"], F32(case.eps)), case.dtype)
    say("checkpointing backward %s shape=%s" % (case.id, (case.N, case.C, case.HW)))
    D = Dev(inp)
    xh = to_device(xh_store, case.dtype)
    g = to_device(inp.dz, case.dtype)
    iabn.iabn_ckpt_backward(xh, g, D.gamma, D.beta, torch.from_numpy(var32).cuda(), D.dgamma,
                            D.dbeta, case.eps, case.slope, workspace=D.ws)
    torch.cuda.synchronize()
    dz64 = f64(inp.dz, case.dtype)
    ref = oracle.backward_from_xhat(f64(xh_store, case.dtype), dz64, inp.gamma, inp.beta, var32,
                                    F32(case.eps), F32(case.slope))
    A = np.abs(inp.gamma) / np.sqrt(var32.astype(np.float64) + F32(case.eps))
    check_grads(D, to_f64(g), ref, case.dtype, scale=float(A.max() * np.abs(dz64).max()))
    assert torch.equal(xh, to_device(xh_store, case.dtype))


# ---------------------------------------------------------------- chains


def _kink_flips(z_gpu, z_ref, slope, dtype, ybound=None, neg_gpu=None):
    """Elements on the other branch than the oracle's: only at the kink.  With
    ``ybound`` (the checkpointing's |y| perturbation from the stored xhat),
    every element within it of the kink may flip.  ``neg_gpu``: the GPU's
    branch where it is not the sign of its stored z (the checkpointing decides
    on y = fma(xhat, gamma, beta), whose sign a stored z loses when a*y
    underflows to -0)."""
    if neg_gpu is None:
        neg_gpu = ~(z_gpu >= 0)
    flip = neg_gpu != ~(z_ref >= 0)
    if flip.any():
        y = np.where(z_ref >= 0, z_ref, z_ref / F32(slope))
        bound = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-2}[dtype] * np.abs(y).max()
        if ybound is None:
            assert np.all(np.abs(y[flip]) <= bound), "branch flips away from the kink"
            assert flip.sum() <= max(8, 1e-5 * flip.size)
        else:
            assert np.all(np.abs(y[flip]) <= np.minimum(bound, ybound[flip] + 1e-6 * np.abs(y).max())), \
                "branch flips away from the kink"
    return flip


@pytest.mark.parametrize("case", CHAIN_CASES, ids=lambda c: c.id)
def test_std_chain_parity(case):
    """Standard forward then standard backward against the oracle's chain."""
    inp = make_inputs(case)
    say("standard chain %s" % case.id)
    D = Dev(inp)
    x = to_device(inp.x, case.dtype)
    z = torch.empty_like(x)
    g = to_device(inp.dz, case.dtype)
    iabn.iabn_std_forward_train(x, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, case.eps,
                                case.momentum, case.slope, workspace=D.ws)
    iabn.iabn_std_backward(x, z, g, D.gamma, D.beta, D.mean, D.var, D.dgamma, D.dbeta, case.eps,
                           case.slope, workspace=D.ws)
    torch.cuda.synchronize()
    fw = oracle_forward(case, inp)
    dz = f64(inp.dz, case.dtype)
    bw = oracle.backward_standard(f64(inp.x, case.dtype), dz, inp.gamma, inp.beta, fw["mean"],
                                  fw["var"], F32(case.eps), F32(case.slope), z=fw["z"])
    flip = _kink_flips(to_f64(z), fw["z"], case.slope, case.dtype)
    # xhat comes from the unrounded x here, so only the kink allowance applies
    # (the storage-rounding terms of the InPlace-ABN chain are an upper bound).
    allow = chain_allowances(fw["z"], dz, bw, fw["var"], inp.gamma, inp.beta, case.eps,
                             case.slope, case.dtype, flip)
    check_chain(to_f64(g), to_f64(D.dgamma), to_f64(D.dbeta), bw, allow, flip, case.dtype)
    # The backward against the oracle's on the forward's own x, z and statistics.
    same = oracle.backward_standard(f64(inp.x, case.dtype), dz, inp.gamma, inp.beta, to_f64(D.mean),
                                    to_f64(D.var), F32(case.eps), F32(case.slope), z=to_f64(z))
    check_same_inputs(to_f64(g), to_f64(D.dgamma), to_f64(D.dbeta), same, case.dtype)


@pytest.mark.parametrize("case", CHAIN_CASES, ids=lambda c: c.id)
def test_ckpt_chain_parity(case):
    """Checkpointing forward, recompute, backward against the oracle's chain;
    the stored xhat carries the storage type's rounding."""
    inp = make_inputs(case)
    say("checkpointing chain %s" % case.id)
    D = Dev(inp)
    xh = to_device(inp.x, case.dtype)
    z = torch.empty_like(xh)
    g = to_device(inp.dz, case.dtype)
    iabn.iabn_ckpt_forward_train(xh, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, case.eps,
                                 case.momentum, case.slope, workspace=D.ws)
    z2 = torch.empty_like(z)
    iabn.iabn_ckpt_recompute(xh, z2, D.gamma, D.beta, case.slope)
    iabn.iabn_ckpt_backward(xh, g, D.gamma, D.beta, D.var, D.dgamma, D.dbeta, case.eps, case.slope,
                            workspace=D.ws)
    torch.cuda.synchronize()
    assert torch.equal(z2, z)
    fw = oracle_forward(case, inp)
    dz = f64(inp.dz, case.dtype)
    xh_ref = oracle.normalize(f64(inp.x, case.dtype), fw["mean"], fw["var"], F32(case.eps))
    bw = oracle.backward_from_xhat(xh_ref, dz, inp.gamma, inp.beta, fw["var"], F32(case.eps),
                                   F32(case.slope))
    flip = _kink_flips(to_f64(z), fw["z"], case.slope, case.dtype,
                       ybound=ckpt_z_slack(xh_ref, inp.gamma, 1.0, case.dtype),
                       neg_gpu=ckpt_branch(to_f64(xh), inp.gamma, inp.beta))
    # Storage rounding of xhat: |xhat_stored - xhat| <= u |xhat|; in the
    # InPlace-ABN allowance that perturbation enters as delta through y, so pass
    # an equivalent z whose recovered xhat error bound covers u |xhat|.
    gam = np.abs(inp.gamma)[None, :, None]
    y_equiv = np.abs(xh_ref) * gam + np.abs(inp.beta)[None, :, None]
    z_equiv = np.where(fw["z"] >= 0, 1.0, -F32(case.slope)) * y_equiv
    allow = chain_allowances(z_equiv, dz, bw, fw["var"], inp.gamma, np.zeros_like(inp.beta),
                             case.eps, case.slope, case.dtype, flip)
    check_chain(to_f64(g), to_f64(D.dgamma), to_f64(D.dbeta), bw, allow, flip, case.dtype)
    # The backward against the oracle's on the forward's own stored xhat and sigma^2.
    same = oracle.backward_from_xhat(to_f64(xh), dz, inp.gamma, inp.beta, to_f64(D.var),
                                     F32(case.eps), F32(case.slope))
    check_same_inputs(to_f64(g), to_f64(D.dgamma), to_f64(D.dbeta), same, case.dtype)


# ---------------------------------------------------------------- full size, sampled


@pytest.mark.parametrize("layer", [0, 7])
def test_backbone_layer_arms_sampled(layer):
    """Full-size backbone layers (fp16, N=8) through every arm's entry points,
    as the benchmark times them; the oracle checks sampled channels."""
    w = workloads.WORKLOADS[5]
    N, C, HW = w.layers[layer]
    inp = workloads.workload_layer(w, layer)
    rng = np.random.default_rng(100 + layer)
    chans = np.unique(np.concatenate([[0, C - 1], rng.choice(C, 6, replace=False)]))
    say("backbone arms layer %d shape=%s channels=%s" % (layer, (N, C, HW), chans.tolist()))
    sub = lambda a: a[:, chans, :]  # noqa: E731
    x64 = f64(sub(inp.x), w.dtype)
    dz64 = f64(sub(inp.dz), w.dtype)
    gc, bc = inp.gamma[chans], inp.beta[chans]
    fw = oracle.forward_train(x64, gc, bc, inp.running_mean[chans], inp.running_var[chans],
                              F32(w.eps), F32(w.momentum), F32(w.slope))
    # standard
    D = Dev(inp)
    x = to_device(inp.x, w.dtype)
    z = torch.empty_like(x)
    g = to_device(inp.dz, w.dtype)
    iabn.iabn_std_forward_train(x, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, w.eps, w.momentum,
                                w.slope, workspace=D.ws)
    iabn.iabn_std_backward(x, z, g, D.gamma, D.beta, D.mean, D.var, D.dgamma, D.dbeta, w.eps,
                           w.slope, workspace=D.ws)
    torch.cuda.synchronize()
    zc = to_f64(z[:, chans])
    assert_close("standard z", zc, fw["z"], w.dtype)
    bw = oracle.backward_standard(x64, dz64, gc, bc, fw["mean"], fw["var"], F32(w.eps), F32(w.slope),
                                  z=fw["z"])
    flip = _kink_flips(zc, fw["z"], w.slope, w.dtype)
    allow = chain_allowances(fw["z"], dz64, bw, fw["var"], gc, bc, w.eps, w.slope, w.dtype, flip)
    check_chain(to_f64(g[:, chans]), to_f64(D.dgamma)[chans], to_f64(D.dbeta)[chans], bw, allow,
                flip, w.dtype)
    same = oracle.backward_standard(x64, dz64, gc, bc, to_f64(D.mean)[chans], to_f64(D.var)[chans],
                                    F32(w.eps), F32(w.slope), z=zc)
    check_same_inputs(to_f64(g[:, chans]), to_f64(D.dgamma)[chans], to_f64(D.dbeta)[chans], same,
                      w.dtype)
    # checkpointing
    D = Dev(inp)
    xh = to_device(inp.x, w.dtype)
    z = torch.empty_like(xh)
    g = to_device(inp.dz, w.dtype)
    iabn.iabn_ckpt_forward_train(xh, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, w.eps,
                                 w.momentum, w.slope, workspace=D.ws)
    z2 = torch.empty_like(z)
    iabn.iabn_ckpt_recompute(xh, z2, D.gamma, D.beta, w.slope)
    iabn.iabn_ckpt_backward(xh, g, D.gamma, D.beta, D.var, D.dgamma, D.dbeta, w.eps, w.slope,
                            workspace=D.ws)
    torch.cuda.synchronize()
    assert torch.equal(z2, z)
    xh_ref = oracle.normalize(x64, fw["mean"], fw["var"], F32(w.eps))
    assert_close("checkpointing xhat", to_f64(xh[:, chans]), xh_ref, w.dtype)
    zc = to_f64(z[:, chans])
    assert_close_slack("checkpointing z", zc, fw["z"], w.dtype,
                       ckpt_z_slack(xh_ref, gc, w.slope, w.dtype))
    bw = oracle.backward_from_xhat(xh_ref, dz64, gc, bc, fw["var"], F32(w.eps), F32(w.slope))
    flip = _kink_flips(zc, fw["z"], w.slope, w.dtype, ybound=ckpt_z_slack(xh_ref, gc, 1.0, w.dtype),
                       neg_gpu=ckpt_branch(to_f64(xh[:, chans]), gc, bc))
    gam = np.abs(gc)[None, :, None]
    z_equiv = np.where(fw["z"] >= 0, 1.0, -F32(w.slope)) * (np.abs(xh_ref) * gam + np.abs(bc)[None, :, None])
    allow = chain_allowances(z_equiv, dz64, bw, fw["var"], gc, np.zeros_like(bc), w.eps, w.slope,
                             w.dtype, flip)
    check_chain(to_f64(g[:, chans]), to_f64(D.dgamma)[chans], to_f64(D.dbeta)[chans], bw, allow,
                flip, w.dtype)
    same = oracle.backward_from_xhat(to_f64(xh[:, chans]), dz64, gc, bc, to_f64(D.var)[chans],
                                     F32(w.eps), F32(w.slope))
    check_same_inputs(to_f64(g[:, chans]), to_f64(D.dgamma)[chans], to_f64(D.dbeta)[chans], same,
                      w.dtype)
    # InPlace-ABN II, from the InPlace-ABN forward's z
    D = Dev(inp)
    xz = to_device(inp.x, w.dtype)
    g = to_device(inp.dz, w.dtype)
    iabn.iabn_forward_train(xz, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, w.eps, w.momentum,
                            w.slope, workspace=D.ws)
    iabn.iabn_backward_ii(xz, g, D.gamma, D.beta, D.var, D.dgamma, D.dbeta, w.eps, w.slope,
                          workspace=D.ws)
    torch.cuda.synchronize()
    zc = to_f64(xz[:, chans])
    bw = oracle.backward_ii(fw["z"], dz64, gc, bc, fw["var"], F32(w.eps), F32(w.slope))
    flip = _kink_flips(zc, fw["z"], w.slope, w.dtype)
    allow = chain_allowances(fw["z"], dz64, bw, fw["var"], gc, bc, w.eps, w.slope, w.dtype, flip)
    check_chain(to_f64(g[:, chans]), to_f64(D.dgamma)[chans], to_f64(D.dbeta)[chans], bw, allow,
                flip, w.dtype)
    same = oracle.backward_ii(zc, dz64, gc, bc, to_f64(D.var)[chans], F32(w.eps), F32(w.slope))
    check_same_inputs(to_f64(g[:, chans]), to_f64(D.dgamma)[chans], to_f64(D.dbeta)[chans], same,
                      w.dtype)


# ---------------------------------------------------------------- determinism and errors


@pytest.mark.parametrize("case", [CONFIG_CASES[3], EDGE_CASES[0]], ids=lambda c: c.id)
def test_arms_deterministic(case):
    inp = make_inputs(case)
    outs = []
    for rep in range(2):
        say("arms determinism %s rep %d" % (case.id, rep))
        D = Dev(inp)
        x = to_device(inp.x, case.dtype)
        z = torch.empty_like(x)
        g = to_device(inp.dz, case.dtype)
        iabn.iabn_std_forward_train(x, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, case.eps,
                                    case.momentum, case.slope, workspace=D.ws)
        iabn.iabn_std_backward(x, z, g, D.gamma, D.beta, D.mean, D.var, D.dgamma, D.dbeta,
                               case.eps, case.slope, workspace=D.ws)
        xh = to_device(inp.x, case.dtype)
        zc = torch.empty_like(xh)
        gc = to_device(inp.dz, case.dtype)
        dg2 = torch.empty_like(D.dgamma)
        db2 = torch.empty_like(D.dbeta)
        iabn.iabn_ckpt_forward_train(xh, zc, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, case.eps,
                                     case.momentum, case.slope, workspace=D.ws)
        iabn.iabn_ckpt_backward(xh, gc, D.gamma, D.beta, D.var, dg2, db2, case.eps, case.slope,
                                workspace=D.ws)
        torch.cuda.synchronize()
        outs.append([z, g, D.dgamma, D.dbeta, xh, zc, gc, dg2, db2])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_arms_errors_leave_outputs_untouched():
    case = EDGE_CASES[0]
    inp = make_inputs(case)
    D = Dev(inp)
    x = to_device(inp.x, case.dtype)
    z = torch.full_like(x, 5.0)
    say("arms error paths")
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_std_forward_train(x, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, 1e-5, 0.1,
                                    -0.5, workspace=D.ws)
    assert e.value.status == 3
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_ckpt_forward_train(x, z, D.gamma, D.beta, D.rm, D.rv, D.mean, D.var, 1e-5, 2.0,
                                     0.01, workspace=D.ws)
    assert e.value.status == 3
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_ckpt_recompute(x, z, D.gamma, D.beta, 0.0)
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert torch.equal(x, to_device(inp.x, case.dtype))
    assert torch.all(z == 5.0)

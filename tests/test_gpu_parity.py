"""GPU parity: libiabn through its C ABI against the double-precision oracle.

Inputs come from the seeded generator (``workloads``) and reach both sides
bit-identically in their storage format; expected values come only from
``oracle``.  Gates (max relative error with a floor of 1e-3 * max|ref|):
1e-4 for fp32 storage, 2e-2 for fp16/bf16 storage with fp32 arithmetic.

Each comparison runs through both ways into the library: the fused entry
points (iabn_forward_train / iabn_backward, which use the channel-resident
kernels when every channel gets its own block) and the phase entry points
(stats + apply, reduce + apply: the streaming kernels).

Three kinds of comparison:
  forward      GPU training forward vs oracle forward on the same x.
  backward     GPU backward vs oracle backward on the same stored z (the
               oracle's z rounded to the storage type), dz and sigma^2, so both
               sides take the leaky-ReLU branch from identical z values.
  chain        GPU forward then GPU backward vs the oracle's forward then
               backward.  Elements whose y lies within rounding of the kink
               can land on different branches in fp32 and fp64; those are
               checked to be kink elements and excluded from the elementwise
               dx comparison, and their contribution bounds the dgamma/dbeta
               comparison.
"""

from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_1712_02616_amd as iabn
import workloads
from chain_allowance import (STORE_ABS, STORE_U, chain_allowances, check_chain,  # noqa: F401
                             check_same_inputs)
from gpu_helpers import GpuLayer, TORCH_DTYPES, TOL, assert_close, max_rel, say, to_device, to_f64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a HIP GPU")]

F32 = lambda v: float(np.float32(v))  # noqa: E731  the value the library sees


@dataclasses.dataclass(frozen=True)
class Case:
    id: str
    N: int
    C: int
    HW: int
    dtype: str
    seed: int
    dz_std: float = 1.0
    gamma_sign: bool = False
    slope: float = 0.01
    eps: float = 1e-5
    momentum: float = 0.1
    beta_shift: float = 0.0  # added to every beta (all-positive / all-negative channels)
    x_shift: float = 0.0  # added to every x (large channel means)


W = workloads.WORKLOADS
CONFIG_CASES = [
    Case("cfg1_tiny_f32", 2, 16, 64, "f32", W[1].seed, dz_std=1.0),
    Case("cfg2_resnet_f32", 32, 256, 3136, "f32", W[2].seed, dz_std=0.1),
    Case("cfg3_segcrop_f16", 4, 256, 36864, "f16", W[3].seed, dz_std=0.1, gamma_sign=True),
    Case("cfg4_wide_bf16", 16, 2048, 784, "bf16", W[4].seed, dz_std=1.0),
]
EDGE_CASES = [
    Case("odd_hw49_f32", 3, 5, 49, "f32", 11, gamma_sign=True),
    Case("odd_hw49_f16", 3, 5, 49, "f16", 12, gamma_sign=True),
    Case("odd_hw49_bf16", 3, 5, 49, "bf16", 13, gamma_sign=True),
    Case("hw1_f32", 7, 6, 1, "f32", 14),
    Case("n1_m2_f16", 1, 3, 2, "f16", 15),
    Case("c1_f32", 5, 1, 1000, "f32", 16),
    Case("ragged_slices_f16", 3, 4, 20008, "f16", 17, dz_std=0.1),
    Case("ragged_slices_bf16", 3, 4, 20008, "bf16", 18, dz_std=0.1),
    Case("ragged_odd_f32", 4, 3, 12345, "f32", 19),
    Case("many_slices_f32", 2, 2, 1 << 20, "f32", 20, dz_std=0.1),
    # Slices of 64K fp16 values on the streaming path (fewer than 256
    # channels): the statistics pass with its deeper batches of loads.
    Case("long_slices_f16", 8, 64, 65536, "f16", 42, dz_std=0.1),
    # Long slices with ragged ends: 8.55 accesses per thread, the last slice
    # 8.48 (one batch of 8, then a partial one), and 32.05 per thread, the
    # last slice 31.83 (the backward's reduction takes batches of 8 as well).
    Case("long_ragged_f16", 4, 16, 140000, "f16", 52, dz_std=0.1, gamma_sign=True),
    Case("long_ragged_reduce_bf16", 2, 8, 2100000, "bf16", 53, dz_std=0.1),
    Case("all_negative_f16", 2, 8, 512, "f16", 21, beta_shift=-12.0),
    Case("all_positive_bf16", 2, 8, 512, "bf16", 22, beta_shift=12.0),
    Case("slope1_plain_bn_f32", 4, 8, 256, "f32", 23, slope=1.0),
    Case("slope_half_f16", 4, 8, 256, "f16", 24, slope=0.5),
    Case("large_mean_f32", 8, 16, 1024, "f32", 25, x_shift=1000.0),
    Case("eps_large_bf16", 4, 16, 96, "bf16", 26, eps=0.5),
    Case("momentum_one_f32", 2, 4, 40, "f32", 27, momentum=1.0),
    # Many channels at the strip-addressed fused shapes (a channel is exactly
    # R strips of T accesses), including T = 256 with 16 strips.
    Case("manych_c600_f16", 8, 600, 4096, "f16", 28, dz_std=0.1, gamma_sign=True),
    Case("manych_c1300_bf16", 4, 1300, 8192, "bf16", 29, dz_std=0.1),
    Case("manych_c520_f32", 4, 520, 4096, "f32", 30, dz_std=0.1),
    Case("manych_t256_c512_f16", 16, 512, 2048, "f16", 31, dz_std=0.1),
    # Two channels per forward block (1024-2047 channels of 4096 accesses on
    # rows of whole strips; manych_c1300_bf16 above takes them as well).
    Case("pair_c1536_f32", 8, 1536, 2048, "f32", 54, dz_std=0.1, gamma_sign=True),
    # Several channels per backward block (512, 768 or 1024 channels of 4096
    # accesses on rows of whole strips; manych_t256_c512_f16 takes them too).
    Case("pair_bwd_c512_f32", 8, 512, 2048, "f32", 55, dz_std=0.1, gamma_sign=True),
    Case("pair_bwd_c1024_bf16", 4, 1024, 8192, "bf16", 56, dz_std=0.1),
    Case("triple_bwd_c768_f16", 8, 768, 4096, "f16", 57, dz_std=0.1, gamma_sign=True),
    # Channels of 1025-2048 accesses: the (256, 8) rung, strip-addressed.
    Case("rung256x8_strip_f16", 8, 300, 2048, "f16", 40, dz_std=0.1, gamma_sign=True),
    Case("rung256x8_strip_f32", 4, 264, 2048, "f32", 41),
    # Fewer channels than CUs with channels that fit a block's registers: the
    # channel-resident kernels from 64 channels (forward) and 96 (backward).
    Case("fewch_c128_f16", 8, 128, 4096, "f16", 43, dz_std=0.1, gamma_sign=True),
    Case("fewch_c96_bf16", 4, 96, 16384, "bf16", 44, dz_std=0.1),
    Case("fewch_c64_f32", 16, 64, 1024, "f32", 45),
    Case("fewch_c128_big_f32", 8, 128, 12544, "f32", 46, dz_std=0.1),
    # Rows that are not a multiple of 16 bytes: the channel-resident kernels
    # with 8-, 4- and 2-byte accesses (14x14 and 7x7 maps, and the like),
    # including channels larger than the registers hold.
    Case("narrow8_hw196_f16", 16, 512, 196, "f16", 32, dz_std=0.1, gamma_sign=True),
    Case("narrow4_hw98_bf16", 8, 300, 98, "bf16", 33, dz_std=0.1),
    Case("narrow2_hw49_f16", 32, 256, 49, "f16", 34, dz_std=0.1),
    Case("narrow4_hw49_f32", 8, 2048, 49, "f32", 35),
    Case("narrow8_hw14_f32", 16, 384, 14, "f32", 36),
    Case("narrow2_bigchan_f16", 384, 256, 49, "f16", 37, dz_std=0.1),
    Case("narrow4_rung256_bf16", 64, 300, 98, "bf16", 38, dz_std=0.1),
    Case("narrow4_rung512_f16", 128, 256, 98, "f16", 39, dz_std=0.1),
    Case("narrow8_few_c200_f16", 32, 200, 196, "f16", 47, dz_std=0.1, gamma_sign=True),
    Case("narrow2_few_c256_bf16", 32, 256, 49, "bf16", 48, dz_std=0.1),
    # One wave per channel in the forward (2048+ channels of 1025-2048
    # accesses): general mapping fp32, strips fp16, 8-byte accesses.
    Case("onewave_c2048_f32", 8, 2048, 784, "f32", 49, gamma_sign=True),
    Case("onewave_strip_c2048_f16", 2, 2048, 8192, "f16", 50, dz_std=0.1),
    Case("onewave_narrow8_c2048_f16", 32, 2048, 196, "f16", 51, dz_std=0.1, gamma_sign=True),
]
ALL_CASES = CONFIG_CASES + EDGE_CASES


def make_inputs(case: Case) -> workloads.LayerInputs:
    inp = workloads.make_layer(case.N, case.C, case.HW, case.dtype, case.seed, dz_std=case.dz_std,
                               gamma_sign=case.gamma_sign)
    if case.beta_shift:
        inp.beta = (inp.beta + np.float32(case.beta_shift)).astype(np.float32)
    if case.x_shift:
        x = workloads.storage_to_f64(inp.x, case.dtype) + case.x_shift
        inp.x = workloads.f64_to_storage(x, case.dtype)
    return inp


def oracle_forward(case: Case, inp: workloads.LayerInputs):
    x = workloads.storage_to_f64(inp.x, case.dtype)
    return oracle.forward_train(x, inp.gamma, inp.beta, inp.running_mean, inp.running_var,
                                F32(case.eps), F32(case.momentum), F32(case.slope))


PATHS = ["entry", "phases"]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("case", ALL_CASES, ids=lambda c: c.id)
def test_forward_parity(case, path):
    inp = make_inputs(case)
    say("forward %s %s shape=%s" % (case.id, path, (case.N, case.C, case.HW)))
    L = GpuLayer(inp)
    L.forward_train(case.eps, case.momentum, case.slope, path=path)
    torch.cuda.synchronize()
    ref = oracle_forward(case, inp)
    assert_close("z", to_f64(L.x).reshape(ref["z"].shape), ref["z"], case.dtype)
    for k in ("mean", "var", "running_mean", "running_var"):
        got = to_f64({"mean": L.save_mean, "var": L.save_var, "running_mean": L.running_mean,
                      "running_var": L.running_var}[k])
        # fp32 arithmetic on exact storage values, whatever the storage type
        assert max_rel(got, ref[k]) <= TOL["f32"], k


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("case", ALL_CASES, ids=lambda c: c.id)
def test_backward_parity(case, path):
    inp = make_inputs(case)
    fw = oracle_forward(case, inp)
    z_store = workloads.f64_to_storage(fw["z"], case.dtype)
    var32 = fw["var"].astype(np.float32)
    say("backward %s %s shape=%s" % (case.id, path, (case.N, case.C, case.HW)))
    L = GpuLayer(inp)
    z_dev = to_device(z_store, case.dtype)
    L.backward(case.eps, case.slope, z=z_dev, save_var=torch.from_numpy(var32).cuda(), path=path)
    torch.cuda.synchronize()
    ref = oracle.backward_i(workloads.storage_to_f64(z_store, case.dtype),
                            workloads.storage_to_f64(inp.dz, case.dtype), inp.gamma, inp.beta,
                            var32, F32(case.eps), F32(case.slope))
    assert_close("dx", to_f64(L.dz).reshape(ref["dx"].shape), ref["dx"], case.dtype)
    assert max_rel(to_f64(L.dgamma), ref["dgamma"]) <= TOL[case.dtype], "dgamma"
    assert max_rel(to_f64(L.dbeta), ref["dbeta"]) <= TOL[case.dtype], "dbeta"
    # z is read-only for the backward
    assert torch.equal(z_dev, to_device(z_store, case.dtype))


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("case", ALL_CASES, ids=lambda c: c.id)
def test_chain_parity(case, path):
    """GPU forward then GPU backward, in place, against the oracle's chain."""
    inp = make_inputs(case)
    say("chain %s %s shape=%s" % (case.id, path, (case.N, case.C, case.HW)))
    L = GpuLayer(inp)
    L.forward_train(case.eps, case.momentum, case.slope, path=path)
    L.backward(case.eps, case.slope, path=path)
    torch.cuda.synchronize()
    fw = oracle_forward(case, inp)
    dz = workloads.storage_to_f64(inp.dz, case.dtype)
    bw = oracle.backward_i(fw["z"], dz, inp.gamma, inp.beta, fw["var"], F32(case.eps),
                           F32(case.slope))
    zg = to_f64(L.x).reshape(fw["z"].shape)
    flip = (zg >= 0) != (fw["z"] >= 0)
    if flip.any():
        # Only elements at the kink may land on the other branch: their y is
        # within a few storage ulps of 0 (fp16 can also flush a tiny a*y to -0).
        y = np.where(fw["z"] >= 0, fw["z"], fw["z"] / F32(case.slope))
        ymax = np.abs(y).max()
        bound = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-2}[case.dtype] * ymax
        assert np.all(np.abs(y[flip]) <= bound), "branch flips away from the kink"
        assert flip.sum() <= max(8, 1e-5 * flip.size)
    allow = chain_allowances(fw["z"], dz, bw, fw["var"], inp.gamma, inp.beta, case.eps,
                             case.slope, case.dtype, flip)
    check_chain(to_f64(L.dz).reshape(bw["dx"].shape), to_f64(L.dgamma), to_f64(L.dbeta), bw, allow,
                flip, case.dtype)
    # The backward against the oracle's on the GPU forward's own z and sigma^2.
    same = oracle.backward_i(zg, dz, inp.gamma, inp.beta, to_f64(L.save_var), F32(case.eps),
                             F32(case.slope))
    check_same_inputs(to_f64(L.dz).reshape(bw["dx"].shape), to_f64(L.dgamma), to_f64(L.dbeta), same,
                      case.dtype)


@pytest.mark.parametrize("case", [CONFIG_CASES[0], EDGE_CASES[0], EDGE_CASES[6], CONFIG_CASES[3]] +
                         [c for c in EDGE_CASES if c.id in ("narrow8_hw196_f16", "narrow4_hw98_bf16")],
                         ids=lambda c: c.id)
def test_eval_parity(case):
    inp = make_inputs(case)
    rng = np.random.default_rng(case.seed)
    rm = rng.uniform(-2, 2, case.C).astype(np.float32)
    rv = rng.uniform(0.25, 9, case.C).astype(np.float32)
    say("eval %s" % case.id)
    x = to_device(inp.x, case.dtype)
    iabn.iabn_forward_eval(x, torch.from_numpy(inp.gamma).cuda(), torch.from_numpy(inp.beta).cuda(),
                           torch.from_numpy(rm).cuda(), torch.from_numpy(rv).cuda(), case.eps,
                           case.slope)
    torch.cuda.synchronize()
    ref = oracle.forward_eval(workloads.storage_to_f64(inp.x, case.dtype), inp.gamma, inp.beta, rm,
                              rv, F32(case.eps), F32(case.slope))
    assert_close("z", to_f64(x).reshape(ref.shape), ref, case.dtype)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("case", [CONFIG_CASES[3], CONFIG_CASES[1], EDGE_CASES[0], EDGE_CASES[7]],
                         ids=lambda c: c.id)
def test_deterministic(case, path):
    """Same inputs, same device: bit-identical outputs."""
    inp = make_inputs(case)
    outs = []
    for rep in range(2):
        say("determinism %s %s rep %d" % (case.id, path, rep))
        L = GpuLayer(inp)
        L.forward_train(case.eps, case.momentum, case.slope, path=path)
        z = L.x.clone()
        L.backward(case.eps, case.slope, path=path)
        torch.cuda.synchronize()
        outs.append([z, L.dz, L.save_mean, L.save_var, L.running_mean, L.running_var, L.dgamma,
                     L.dbeta])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("case", [EDGE_CASES[0], EDGE_CASES[7], EDGE_CASES[3]], ids=lambda c: c.id)
def test_phases_equal_entry_on_streaming_shapes(case):
    """Where the entry points take the streaming kernels (few channels, or
    the one-element path), stats+apply and reduce+apply are exactly them."""
    inp = make_inputs(case)
    say("phases %s" % case.id)
    A = GpuLayer(inp)
    A.forward_train(case.eps, case.momentum, case.slope)
    A.backward(case.eps, case.slope)
    B = GpuLayer(inp)
    B.forward_train(case.eps, case.momentum, case.slope, path="phases")
    B.backward(case.eps, case.slope, path="phases")
    torch.cuda.synchronize()
    for k in ("x", "dz", "save_mean", "save_var", "running_mean", "running_var", "dgamma", "dbeta"):
        assert torch.equal(getattr(A, k), getattr(B, k)), k


@pytest.mark.parametrize("dtype,offset,C", [("f32", 16, 6), ("f16", 8, 6), ("bf16", 3, 6), ("f32", 1, 6),
                                            ("f16", 4, 256), ("bf16", 2, 256), ("f32", 2, 256),
                                            ("f16", 1, 256)])
def test_guard_band_and_alignment(dtype, offset, C):
    """Run inside a larger buffer: nothing outside [x, x+E) changes, and an
    offset that breaks 16-byte alignment takes a narrower access (8, 4 or 2
    bytes; with C = 256 on the channel-resident kernels) with the same
    results (to the parity tolerance)."""
    case = Case("guard_%s_%d_c%d" % (dtype, offset, C), 3, C, 800, dtype, 30)
    inp = make_inputs(case)
    N, C, HW = case.N, case.C, case.HW
    E = N * C * HW
    G = 4096  # guard elements after the tensor; `offset` guard elements before it
    tdt = TORCH_DTYPES[dtype]
    say("guard %s offset %d" % (dtype, offset))
    xbuf = torch.full((E + 2 * G,), 7.25, dtype=tdt, device="cuda")
    gbuf = torch.full((E + 2 * G,), -3.5, dtype=tdt, device="cuda")
    x = xbuf[offset: offset + E].view(N, C, HW)
    dz = gbuf[offset: offset + E].view(N, C, HW)
    x.copy_(to_device(inp.x, dtype))
    dz.copy_(to_device(inp.dz, dtype))
    L = GpuLayer(inp)
    iabn.iabn_forward_train(x, L.gamma, L.beta, L.running_mean, L.running_var, L.save_mean,
                            L.save_var, case.eps, case.momentum, case.slope)
    iabn.iabn_backward(x, dz, L.gamma, L.beta, L.save_var, L.dgamma, L.dbeta, case.eps, case.slope)
    torch.cuda.synchronize()
    for buf, fill in ((xbuf, 7.25), (gbuf, -3.5)):
        assert torch.all(buf[:offset] == fill) and torch.all(buf[offset + E:] == fill)
    fw = oracle_forward(case, inp)
    bw = oracle.backward_i(fw["z"], workloads.storage_to_f64(inp.dz, dtype), inp.gamma, inp.beta,
                           fw["var"], F32(case.eps), F32(case.slope))
    assert_close("z", to_f64(x), fw["z"], dtype)
    zg = to_f64(x)
    flip = (zg >= 0) != (fw["z"] >= 0)
    dzf = workloads.storage_to_f64(inp.dz, dtype)
    allow = chain_allowances(fw["z"], dzf, bw, fw["var"], inp.gamma, inp.beta, case.eps, case.slope,
                             dtype, flip)
    check_chain(to_f64(dz), to_f64(L.dgamma), to_f64(L.dbeta), bw, allow, flip, dtype)
    same = oracle.backward_i(zg, dzf, inp.gamma, inp.beta, to_f64(L.save_var), F32(case.eps),
                             F32(case.slope))
    check_same_inputs(to_f64(dz), to_f64(L.dgamma), to_f64(L.dbeta), same, dtype)


def test_errors_leave_outputs_untouched():
    case = EDGE_CASES[0]
    inp = make_inputs(case)
    L = GpuLayer(inp)
    before = L.x.clone()
    rm = L.running_mean.clone()
    small = torch.empty(8, dtype=torch.uint8, device="cuda")
    say("error paths")
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_forward_train(L.x, L.gamma, L.beta, L.running_mean, L.running_var, L.save_mean,
                                L.save_var, 1e-5, 0.1, 0.01, workspace=small)
    assert e.value.status == 5
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_forward_train(L.x, L.gamma, L.beta, L.running_mean, L.running_var, L.save_mean,
                                L.save_var, 1e-5, 0.1, 0.0)
    assert e.value.status == 3
    with pytest.raises(iabn.IabnError):
        iabn.iabn_backward(L.x, L.dz, L.gamma, L.beta, L.save_var, L.dgamma, L.dbeta, -1.0, 0.01)
    torch.cuda.synchronize()
    assert torch.equal(L.x, before) and torch.equal(L.running_mean, rm)


# ------------------------------------------------------------ full size, sampled


BACKBONE_GROUPS = [0, 3, 7, 30]  # first layer of each (C, H=W) group of the backbone sweep


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("layer", BACKBONE_GROUPS)
def test_backbone_layer_sampled(layer, path):
    """A full-size layer of the backbone sweep (fp16, N=8) through the same
    entry points the benchmark times; the oracle checks sampled channels,
    each computed on its own (channels are independent)."""
    w = workloads.WORKLOADS[5]
    N, C, HW = w.layers[layer]
    inp = workloads.workload_layer(w, layer)
    rng = np.random.default_rng(layer)
    chans = np.unique(np.concatenate([[0, C - 1], rng.choice(C, 6, replace=False)]))
    say("backbone layer %d %s shape=%s channels=%s" % (layer, path, (N, C, HW), chans.tolist()))
    L = GpuLayer(inp)
    L.forward_train(w.eps, w.momentum, w.slope, path=path)
    L.backward(w.eps, w.slope, path=path)
    torch.cuda.synchronize()
    zc = to_f64(L.x[:, chans])
    dxc = to_f64(L.dz[:, chans])
    sub = lambda a: a[:, chans, :]  # noqa: E731
    x = workloads.storage_to_f64(sub(inp.x), w.dtype)
    dz = workloads.storage_to_f64(sub(inp.dz), w.dtype)
    fw = oracle.forward_train(x, inp.gamma[chans], inp.beta[chans], inp.running_mean[chans],
                              inp.running_var[chans], F32(w.eps), F32(w.momentum), F32(w.slope))
    bw = oracle.backward_i(fw["z"], dz, inp.gamma[chans], inp.beta[chans], fw["var"], F32(w.eps),
                           F32(w.slope))
    assert_close("z", zc, fw["z"], w.dtype)
    for k, got in (("mean", L.save_mean), ("var", L.save_var), ("running_mean", L.running_mean),
                   ("running_var", L.running_var)):
        assert max_rel(to_f64(got)[chans], fw[k]) <= TOL["f32"], k
    flip = (zc >= 0) != (fw["z"] >= 0)
    assert flip.sum() <= max(8, 1e-5 * flip.size)
    allow = chain_allowances(fw["z"], dz, bw, fw["var"], inp.gamma[chans], inp.beta[chans], w.eps,
                             w.slope, w.dtype, flip)
    check_chain(dxc, to_f64(L.dgamma)[chans], to_f64(L.dbeta)[chans], bw, allow, flip, w.dtype)
    same = oracle.backward_i(zc, dz, inp.gamma[chans], inp.beta[chans], to_f64(L.save_var)[chans],
                             F32(w.eps), F32(w.slope))
    check_same_inputs(dxc, to_f64(L.dgamma)[chans], to_f64(L.dbeta)[chans], same, w.dtype)

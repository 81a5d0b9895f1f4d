"""CPU pins of the end-to-end chain allowances (``chain_allowance``): the
allowance must admit what keeping z in 16-bit storage does to an exact
backward, and must not admit a real error.

The chain a perfect device would produce: the exact forward's z rounded to
the storage type, the exact InPlace-ABN I backward from that stored z, dx
rounded to the storage type and dgamma, dbeta to fp32.  Against the exact
chain (the backward from the unrounded z) that passes ``check_chain``; the
same results with dx off by 2.5% or 4% fail it.  The allowance of dgamma is a
worst-case sum over the channel (every rounding of z taken with the sign of
dy*y), loose by design; dgamma and dbeta are held to the gate by the
same-input comparison (``check_same_inputs``: the oracle's backward on the
chain's own stored z), which fails them off by 2.5%, and passes the perfect
device's results."""

from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads
from chain_allowance import F32, chain_allowances, check_chain, check_same_inputs

SHAPES = [  # (N, C, HW, dtype, seed, dz_std)
    (3, 4, 20008, "bf16", 18, 0.1),
    (4, 64, 784, "bf16", 81, 1.0),
    (8, 16, 4096, "f16", 82, 0.1),
    (3, 5, 49, "f16", 12, 1.0),
]
EPS, MOM, SLOPE = 1e-5, 0.1, 0.01


def chains(N, C, HW, dtype, seed, dz_std):
    inp = workloads.make_layer(N, C, HW, dtype, seed, dz_std=dz_std, gamma_sign=True)
    x = workloads.storage_to_f64(inp.x, dtype)
    dz = workloads.storage_to_f64(inp.dz, dtype)
    fw = oracle.forward_train(x, inp.gamma, inp.beta, inp.running_mean, inp.running_var, F32(EPS),
                              F32(MOM), F32(SLOPE))
    exact = oracle.backward_i(fw["z"], dz, inp.gamma, inp.beta, fw["var"], F32(EPS), F32(SLOPE))
    zs = workloads.storage_to_f64(workloads.f64_to_storage(fw["z"], dtype), dtype)
    stored = oracle.backward_i(zs, dz, inp.gamma, inp.beta, fw["var"], F32(EPS), F32(SLOPE))
    dx = workloads.storage_to_f64(workloads.f64_to_storage(stored["dx"], dtype), dtype)
    dg = stored["dgamma"].astype(np.float32).astype(np.float64)
    db = stored["dbeta"].astype(np.float32).astype(np.float64)
    flip = (zs >= 0) != (fw["z"] >= 0)
    allow = chain_allowances(fw["z"], dz, exact, fw["var"], inp.gamma, inp.beta, EPS, SLOPE, dtype,
                             flip)
    return exact, (dx, dg, db), allow, flip, stored


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%dx%d_%s" % s[:4])
def test_stored_z_chain_passes(shape):
    exact, (dx, dg, db), allow, flip, stored = chains(*shape)
    check_chain(dx, dg, db, exact, allow, flip, shape[3])
    check_same_inputs(dx, dg, db, stored, shape[3])


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%dx%d_%s" % s[:4])
@pytest.mark.parametrize("factor", [1.025, 1.04, 0.975])
def test_planted_dx_error_fails_the_allowance(shape, factor):
    exact, (dx, dg, db), allow, flip, stored = chains(*shape)
    with pytest.raises(AssertionError):
        check_chain(dx * factor, dg, db, exact, allow, flip, shape[3])


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%dx%d_%s" % s[:4])
@pytest.mark.parametrize("what", ["dx", "dgamma", "dbeta"])
def test_planted_error_fails_the_same_input_check(shape, what):
    exact, (dx, dg, db), allow, flip, stored = chains(*shape)
    got = {"dx": dx, "dgamma": dg, "dbeta": db}
    got[what] = got[what] * 1.025
    with pytest.raises(AssertionError):
        check_same_inputs(got["dx"], got["dgamma"], got["dbeta"], stored, shape[3])

"""The allowances of the end-to-end chain comparison (GPU forward, then GPU
backward from the GPU's own stored z, against the oracle's exact chain):
what keeping z in the storage type provably moves the backward's results by,
and the check that applies them.  numpy only, shared by the GPU parity tests
and pinned on the CPU by ``test_chain_allowance.py``."""

from __future__ import annotations

import numpy as np

from gpu_helpers import TOL

F32 = lambda v: float(np.float32(v))  # noqa: E731  the value the library sees


# Unit roundoff of the stored z, plus a few fp32 roundings of the kernel's y
# before the store; and the absolute half-ulp below which a*y flushes into
# fp16 subnormals / zero.
STORE_U = {"f32": 4 * 2.0 ** -24, "f16": 2.0 ** -11 + 4 * 2.0 ** -24,
           "bf16": 2.0 ** -8 + 4 * 2.0 ** -24}
STORE_ABS = {"f32": 2.0 ** -150, "f16": 2.0 ** -25, "bf16": 2.0 ** -134}


def chain_allowances(z_ref, dz, ref, var, gamma, beta, eps, slope, dtype, flip):
    """What a forward + backward chain with z kept in the storage type may
    differ from the exact-arithmetic chain by, beyond the tolerance.

    - Elements that took the other branch at the kink (``flip``) change dbeta
      by (1 - a) dz_i and dgamma by (1 - a) dz_i xhat_i, with |y_i| <= 1 there.
    - The backward recovers xhat from the stored z.  With unit roundoff u of
      the storage type, |y_stored - y| <= u |y| + h/a (h: half the smallest
      subnormal step), so delta_i = |xhat_stored_i - xhat_i| <= (u |y_i| + h/a)/|gamma|,
      dgamma = sum dy xhat moves by at most D = sum |dy_i| delta_i, and
      dx_i = A (dy_i - dgamma xhat_i/m - dbeta/m) by at most
      |A|/m (|dgamma| delta_i + D (|xhat_i| + delta_i)) (first order).
    Returns (dx, dgamma, dbeta) allowances.
    """
    g = np.asarray(gamma, np.float64)[None, :, None]
    b = np.asarray(beta, np.float64)[None, :, None]
    a = F32(slope)
    m = z_ref.shape[0] * z_ref.shape[2]
    y = np.where(z_ref >= 0, z_ref, z_ref / a)
    dy = np.where(z_ref >= 0, dz, a * dz)
    xhat = (y - b) / g
    delta = (STORE_U[dtype] * np.abs(y) + STORE_ABS[dtype] / a) / np.abs(g)
    flipped = np.abs(np.where(flip, dz, 0.0))
    slack_b = flipped.sum(axis=(0, 2))
    slack_g = (flipped * (np.abs(b) + 1.0) / np.abs(g)).sum(axis=(0, 2))
    D = (np.abs(dy) * delta).sum(axis=(0, 2))
    slack_g = slack_g + D
    A = np.abs(g) / np.sqrt(np.asarray(var, np.float64)[None, :, None] + F32(eps))
    dg = np.abs(ref["dgamma"])[None, :, None]
    slack_dx = A / m * (dg * delta + (D + slack_b)[None, :, None] * (np.abs(xhat) + delta + 1.0))
    return slack_dx, slack_g, slack_b


def check_chain(dx, dgamma, dbeta, ref, allow, flip, dtype, scales=None):
    """``scales``: the max |ref| of dx, dgamma and dbeta over the whole tensor
    when ``ref`` covers only some of its channels (the relative error's floor
    is 1e-3 of that); by default the maxima over ``ref`` itself."""
    slack_dx, slack_g, slack_b = allow
    keep = ~flip
    sc = scales or {k: np.abs(ref[k]).max() for k in ("dx", "dgamma", "dbeta")}
    floor = np.maximum(np.abs(ref["dx"]), 1e-3 * sc["dx"])
    err = np.abs(dx - ref["dx"]) - slack_dx
    assert np.all(np.isfinite(dx)), "dx has non-finite values"
    worst = float(np.max((err / floor)[keep])) if keep.any() else 0.0
    assert worst <= TOL[dtype], "dx: max rel err beyond allowance %.3e > %.1e" % (worst, TOL[dtype])
    for name, got, r, slack in (("dbeta", dbeta, ref["dbeta"], slack_b),
                                ("dgamma", dgamma, ref["dgamma"], slack_g)):
        fl = np.maximum(np.abs(r), 1e-3 * sc[name])
        bad = np.abs(got - r) > TOL[dtype] * fl + slack
        assert not bad.any(), "%s: channels %s got %s ref %s slack %s" % (
            name, np.nonzero(bad)[0][:5], got[bad][:5], r[bad][:5], slack[bad][:5])


def check_same_inputs(dx, dgamma, dbeta, ref, dtype, scales=None):
    """A chain's backward against the oracle's backward run on the chain's
    own stored tensors and saved statistics (the GPU forward's z, or xhat,
    and its fp32 sigma^2): both sides start from identical inputs, so no
    allowance applies, only the gate (relative error floored at 1e-3 of the
    maximum, over the whole tensor when ``scales`` gives its maxima)."""
    sc = scales or {k: np.abs(ref[k]).max() for k in ("dx", "dgamma", "dbeta")}
    for name, got in (("dx", dx), ("dgamma", dgamma), ("dbeta", dbeta)):
        got = np.asarray(got, np.float64)
        r = ref[name]
        assert np.all(np.isfinite(got)), "%s has non-finite values" % name
        err = float(np.max(np.abs(got - r) / np.maximum(np.abs(r), 1e-3 * sc[name]))) if r.size else 0.0
        assert err <= TOL[dtype], "%s (same inputs): max rel err %.3e > %.1e" % (name, err, TOL[dtype])

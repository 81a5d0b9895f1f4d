"""Pins for the double-precision oracle (CPU only).

Each test ties the oracle to something other than itself: exact rational
arithmetic, closed forms, invariants that the paper's definitions imply,
central finite differences of the forward, an independent library
implementation (PyTorch's float64 batch_norm + leaky_relu with autograd), and
agreement between the paper's algebraically equivalent backward formulations.
"""

from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import workloads

EPS = 1e-5
SLOPE = 0.01


def _random_layer(N, C, HW, seed, gamma_sign=False, dz_std=1.0):
    inp = workloads.make_layer(N, C, HW, "f32", seed, dz_std=dz_std, gamma_sign=gamma_sign)
    return (workloads.storage_to_f64(inp.x, "f32"), workloads.storage_to_f64(inp.dz, "f32"),
            inp.gamma.astype(np.float64), inp.beta.astype(np.float64))


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------- statistics


def test_batch_stats_exact_rational():
    """Mean and biased variance (Sec. 3.1) against exact rational arithmetic."""
    rng = np.random.default_rng(5)
    N, C, HW = 3, 4, 7
    x = rng.integers(-4000, 4000, size=(N, C, HW)) / 64.0  # dyadic, exact in double
    mean, var = oracle.batch_stats(x)
    m = N * HW
    for c in range(C):
        vals = [Fraction(float(v)) for v in x[:, c, :].ravel()]
        mu = sum(vals) / m
        s2 = sum((v - mu) ** 2 for v in vals) / m
        assert abs(Fraction(mean[c]) - mu) <= abs(mu) * Fraction(1, 2 ** 51) + Fraction(1, 2 ** 60)
        assert abs(Fraction(var[c]) - s2) <= s2 * Fraction(1, 2 ** 50)


def test_batch_stats_arithmetic_sequence_closed_form():
    """x_j = a + h*j over a channel's m values: mu = a + h(m-1)/2, sigma^2 = h^2(m^2-1)/12."""
    N, C, HW = 4, 3, 25
    m = N * HW
    a = np.array([-3.0, 0.5, 1e3])
    h = np.array([0.25, 1.5, 1e-3])
    x = np.empty((N, C, HW))
    for c in range(C):
        x[:, c, :] = (a[c] + h[c] * np.arange(m)).reshape(N, HW)
    mean, var = oracle.batch_stats(x)
    np.testing.assert_allclose(mean, a + h * (m - 1) / 2, rtol=1e-14)
    np.testing.assert_allclose(var, h * h * (m * m - 1) / 12, rtol=1e-12)


def test_batch_stats_matches_numpy():
    x, _, _, _ = _random_layer(5, 6, 33, seed=11)
    mean, var = oracle.batch_stats(x)
    np.testing.assert_allclose(mean, x.mean(axis=(0, 2)), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(var, x.var(axis=(0, 2)), rtol=1e-13)


# ---------------------------------------------------------------- forward


def test_forward_exact_worked_example():
    """One channel x = (2, 2, 4, 4): mu = 3, sigma^2 = 1.  With eps = 2^-9 + 2^-20,
    sqrt(sigma^2 + eps) = 1 + 2^-10 exactly, so z is a rational number we can
    compute without rounding.  Dyadic gamma, beta and slope keep it exact."""
    x = np.array([2.0, 2.0, 4.0, 4.0]).reshape(1, 1, 4)
    eps = 2.0 ** -9 + 2.0 ** -20
    gamma, beta, slope = 2.0, 0.5, 0.25
    out = oracle.forward_train(x, [gamma], [beta], [0.0], [1.0], eps, 0.5, slope)
    assert out["mean"][0] == 3.0 and out["var"][0] == 1.0
    denom = Fraction(1) + Fraction(1, 2 ** 10)
    for k, xv in enumerate([2, 2, 4, 4]):
        y = Fraction(int(gamma)) * (Fraction(xv) - 3) / denom + Fraction(1, 2)
        z = y if y >= 0 else Fraction(1, 4) * y
        assert abs(Fraction(out["z"][0, 0, k]) - z) <= abs(z) * Fraction(1, 2 ** 51)
    # running stats: 0.5*0 + 0.5*3, 0.5*1 + 0.5 * 1 * 4/3
    assert out["running_mean"][0] == 1.5
    assert abs(out["running_var"][0] - (0.5 + 0.5 * 4.0 / 3.0)) < 1e-15


@pytest.mark.parametrize("shape", [(2, 16, 64), (3, 5, 49), (1, 4, 2), (7, 2, 1)])
def test_forward_whitening_invariants(shape):
    """With gamma = 1, beta = 0 and slope 1 the layer returns xhat of Eq. (1):
    per channel sum(xhat) = 0 and mean(xhat^2) = sigma^2 / (sigma^2 + eps)."""
    x, _, _, _ = _random_layer(*shape, seed=3)
    C = shape[1]
    eps = 0.1  # large, so that a dropped eps would show
    out = oracle.forward_train(x, np.ones(C), np.zeros(C), np.zeros(C), np.ones(C), eps, 0.1, 1.0)
    xhat = out["z"]
    var = x.var(axis=(0, 2))
    np.testing.assert_allclose(xhat.mean(axis=(0, 2)), 0.0, atol=1e-13)
    np.testing.assert_allclose((xhat ** 2).mean(axis=(0, 2)), var / (var + eps), rtol=1e-12)


def test_forward_affine_roles():
    """With slope 1: mean(z) = beta and var(z) = gamma^2 sigma^2/(sigma^2+eps) per channel."""
    x, _, g, b = _random_layer(4, 8, 50, seed=4, gamma_sign=True)
    C = 8
    out = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, 1.0)
    var = x.var(axis=(0, 2))
    np.testing.assert_allclose(out["z"].mean(axis=(0, 2)), b, atol=1e-13)
    np.testing.assert_allclose(out["z"].var(axis=(0, 2)), g * g * var / (var + EPS), rtol=1e-12)


def test_forward_shift_and_scale_invariance():
    """BN output does not change when a channel is shifted; scaling x by s and eps
    by s^2 leaves it unchanged too."""
    x, _, g, b = _random_layer(2, 6, 40, seed=8)
    C = 6
    shift = np.linspace(-50, 50, C)[None, :, None]
    base = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)["z"]
    shifted = oracle.forward_train(x + shift, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)["z"]
    scaled = oracle.forward_train(x * 8.0, g, b, np.zeros(C), np.ones(C), EPS * 64, 0.1, SLOPE)["z"]
    assert _rel(shifted, base) < 1e-12
    assert _rel(scaled, base) < 1e-13


def test_forward_leaky_branch():
    """z < 0 exactly where y < 0, and there z = slope * y (Sec. 3.3)."""
    x, _, g, b = _random_layer(2, 4, 100, seed=9)
    C = 4
    z = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, 0.2)["z"]
    y = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, 1.0)["z"]
    neg = y < 0
    assert neg.any() and (~neg).any()
    np.testing.assert_array_equal(z < 0, neg)
    np.testing.assert_allclose(z[neg], 0.2 * y[neg], rtol=1e-15)
    np.testing.assert_array_equal(z[~neg], y[~neg])


@pytest.mark.parametrize("momentum", [0.0, 1.0, 0.1, 0.37])
def test_running_statistics(momentum):
    """Running mean/var blend with momentum; the variance is the unbiased one."""
    x, _, g, b = _random_layer(3, 5, 21, seed=12)
    C = 5
    rm0 = np.linspace(-1, 1, C)
    rv0 = np.linspace(0.5, 2, C)
    out = oracle.forward_train(x, g, b, rm0, rv0, EPS, momentum, SLOPE)
    mu = x.mean(axis=(0, 2))
    unbiased = x.transpose(1, 0, 2).reshape(C, -1).var(axis=1, ddof=1)
    np.testing.assert_allclose(out["running_mean"], (1 - momentum) * rm0 + momentum * mu,
                               rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(out["running_var"], (1 - momentum) * rv0 + momentum * unbiased,
                               rtol=1e-13)
    if momentum == 0.0:
        np.testing.assert_array_equal(out["running_mean"], rm0)
        np.testing.assert_array_equal(out["running_var"], rv0)


def test_eval_equals_train_with_batch_statistics():
    x, _, g, b = _random_layer(2, 7, 30, seed=13, gamma_sign=True)
    C = 7
    tr = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    ev = oracle.forward_eval(x, g, b, tr["mean"], tr["var"], EPS, SLOPE)
    assert _rel(ev, tr["z"]) < 1e-14


def test_leaky_relu_round_trip():
    """f^-1(f(y)) = y; exact for dyadic slopes, within one rounding otherwise."""
    ys = [-3.5, -1e-300, -0.0, 0.0, 1e-300, 2.75, -123456.789, 7e10]
    for a in (0.5, 2.0 ** -7, 1.0):
        for y in ys:
            assert oracle.leaky_relu_inv(oracle.leaky_relu(y, a), a) == y
    for y in ys:
        r = oracle.leaky_relu_inv(oracle.leaky_relu(y, 0.01), 0.01)
        assert abs(r - y) <= 2 * np.spacing(abs(y)) + 1e-320
    assert oracle.leaky_relu(-2.0, 0.01) == -0.02
    assert oracle.leaky_relu_inv(-0.02, 0.01) == -2.0
    assert oracle.leaky_relu(3.0, 0.01) == 3.0


def test_affine_inversion_round_trip_exact():
    """pi^{-1}(pi(xhat)) = xhat through the oracle's forward and backward with
    gamma = +-2^k, beta = 0 and slope 2^-k: dgamma equals sum(dy * xhat) for the
    true xhat exactly enough to match a hand sum."""
    x, dz, _, _ = _random_layer(2, 2, 16, seed=21)
    g = np.array([4.0, -0.5])
    b = np.zeros(2)
    fw = oracle.forward_train(x, g, b, np.zeros(2), np.ones(2), EPS, 0.1, 0.125)
    bw = oracle.backward_i(fw["z"], dz, g, b, fw["var"], EPS, 0.125)
    xhat = (x - fw["mean"][None, :, None]) / np.sqrt(fw["var"][None, :, None] + EPS)
    dy = np.where(fw["z"] >= 0, dz, 0.125 * dz)
    np.testing.assert_allclose(bw["dgamma"], (dy * xhat).sum(axis=(0, 2)), rtol=1e-13)


# ---------------------------------------------------------------- backward


def _loss(x, dz, g, b, eps, slope):
    C = x.shape[1]
    z = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), eps, 0.1, slope)["z"]
    return float(np.sum(dz * z))


def _fd_inputs(seed):
    """Config-1-like tiny layer whose y values stay clear of the kink at 0."""
    for s in range(seed, seed + 50):
        x, dz, g, b = _random_layer(2, 3, 6, seed=s, gamma_sign=True)
        C = 3
        y = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, 1.0)["z"]
        if np.min(np.abs(y)) > 1e-3:
            return x, dz, g, b
    raise AssertionError("no kink-free draw")


def test_backward_i_finite_differences():
    """dL/dx, dL/dgamma, dL/dbeta of L = sum(dz * z(x; gamma, beta)) by central
    differences, against InPlace-ABN I computed from z alone."""
    x, dz, g, b = _fd_inputs(100)
    C = x.shape[1]
    fw = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    bw = oracle.backward_i(fw["z"], dz, g, b, fw["var"], EPS, SLOPE)
    h = 1e-6
    fd = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        xp = x.copy()
        xp[idx] += h
        xm = x.copy()
        xm[idx] -= h
        fd[idx] = (_loss(xp, dz, g, b, EPS, SLOPE) - _loss(xm, dz, g, b, EPS, SLOPE)) / (2 * h)
    assert _rel(bw["dx"], fd) < 1e-6
    fdg = np.zeros(C)
    fdb = np.zeros(C)
    for c in range(C):
        e = np.zeros(C)
        e[c] = h
        fdg[c] = (_loss(x, dz, g + e, b, EPS, SLOPE) - _loss(x, dz, g - e, b, EPS, SLOPE)) / (2 * h)
        fdb[c] = (_loss(x, dz, g, b + e, EPS, SLOPE) - _loss(x, dz, g, b - e, EPS, SLOPE)) / (2 * h)
    assert _rel(bw["dgamma"], fdg) < 1e-6
    assert _rel(bw["dbeta"], fdb) < 1e-6


@pytest.mark.parametrize("shape,seed,gsign", [((2, 16, 64), 1, False), ((4, 9, 49), 2, True),
                                              ((1, 3, 2), 3, True), ((6, 2, 1), 4, False)])
def test_backward_formulations_agree(shape, seed, gsign):
    """InPlace-ABN I (from z via xhat), InPlace-ABN II (from y) and the standard
    chain-rule backward from the stored x are the same gradient (Sec. 3.3, Appendix)."""
    x, dz, g, b = _random_layer(*shape, seed=seed, gamma_sign=gsign)
    C = shape[1]
    fw = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    i = oracle.backward_i(fw["z"], dz, g, b, fw["var"], EPS, SLOPE)
    ii = oracle.backward_ii(fw["z"], dz, g, b, fw["var"], EPS, SLOPE)
    st = oracle.backward_standard(x, dz, g, b, fw["mean"], fw["var"], EPS, SLOPE)
    for k in ("dx", "dgamma", "dbeta"):
        assert _rel(ii[k], i[k]) < 1e-11, k
        assert _rel(st[k], i[k]) < 1e-11, k


def test_backward_invariants():
    """Per channel: sum_i dx_i = 0; sum_i dx_i xhat_i = A dgamma eps/(sigma^2+eps)
    with A = gamma/sqrt(sigma^2+eps); dbeta = sum_{z>=0} dz + a sum_{z<0} dz."""
    x, dz, g, b = _random_layer(3, 5, 40, seed=31, gamma_sign=True)
    C = 5
    eps = 0.05
    fw = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), eps, 0.1, SLOPE)
    bw = oracle.backward_i(fw["z"], dz, g, b, fw["var"], eps, SLOPE)
    scale = np.abs(bw["dx"]).max()
    np.testing.assert_allclose(bw["dx"].sum(axis=(0, 2)), 0.0, atol=1e-12 * scale * x[:, 0].size)
    var = fw["var"]
    xhat = (x - fw["mean"][None, :, None]) / np.sqrt(var[None, :, None] + eps)
    A = g / np.sqrt(var + eps)
    np.testing.assert_allclose((bw["dx"] * xhat).sum(axis=(0, 2)), A * bw["dgamma"] * eps / (var + eps),
                               rtol=1e-9, atol=1e-12)
    pos = fw["z"] >= 0
    db = np.where(pos, dz, 0.0).sum(axis=(0, 2)) + SLOPE * np.where(pos, 0.0, dz).sum(axis=(0, 2))
    np.testing.assert_allclose(bw["dbeta"], db, rtol=1e-13)


@pytest.mark.parametrize("slope", [0.01, 0.3, 1.0])
def test_against_torch_float64_autograd(slope):
    """PyTorch's own float64 batch_norm (training mode: biased variance for the
    normalisation, unbiased variance and momentum for the running estimate) and
    leaky_relu, differentiated by autograd, as an independent implementation."""
    x, dz, g, b = _random_layer(4, 6, 30, seed=41, gamma_sign=True)
    C = 6
    rm0 = np.linspace(-0.5, 0.5, C)
    rv0 = np.linspace(0.5, 1.5, C)
    fw = oracle.forward_train(x, g, b, rm0, rv0, EPS, 0.1, slope)
    bw = oracle.backward_i(fw["z"], dz, g, b, fw["var"], EPS, slope)

    tx = torch.tensor(x.reshape(4, C, 5, 6), requires_grad=True)
    tg = torch.tensor(g, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    trm = torch.tensor(rm0)
    trv = torch.tensor(rv0)
    y = torch.nn.functional.batch_norm(tx, trm, trv, tg, tb, training=True, momentum=0.1, eps=EPS)
    z = torch.nn.functional.leaky_relu(y, slope)
    z.backward(torch.tensor(dz.reshape(4, C, 5, 6)))
    assert _rel(fw["z"], z.detach().numpy().reshape(4, C, 30)) < 1e-13
    np.testing.assert_allclose(fw["running_mean"], trm.numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(fw["running_var"], trv.numpy(), rtol=1e-13)
    assert _rel(bw["dx"], tx.grad.numpy().reshape(4, C, 30)) < 1e-11
    assert _rel(bw["dgamma"], tg.grad.numpy()) < 1e-11
    assert _rel(bw["dbeta"], tb.grad.numpy()) < 1e-11


def test_inplace_aliasing_allowed():
    """The oracle's forward and backward give the same answers when the output
    array is the input array (Algorithm 1 and 2 allow x, y, z and dx, dy, dz to
    share storage)."""
    x, dz, g, b = _random_layer(2, 3, 10, seed=51)
    C = 3
    ref = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    lib = oracle._load()
    buf = x.copy()
    rm, rv = np.zeros(C), np.ones(C)
    mean, var = np.empty(C), np.empty(C)
    P = oracle._ptr
    lib.oracle_forward_train(P(buf), 2, C, 10, P(g.copy()), P(b.copy()), EPS, 0.1, SLOPE, P(rm), P(rv),
                             P(buf), P(mean), P(var))
    np.testing.assert_array_equal(buf, ref["z"])
    bref = oracle.backward_i(ref["z"], dz, g, b, ref["var"], EPS, SLOPE)
    gbuf = dz.copy()
    dg, db = np.empty(C), np.empty(C)
    lib.oracle_backward_i(P(buf), P(gbuf), 2, C, 10, P(g.copy()), P(b.copy()), P(var), EPS, SLOPE,
                          P(gbuf), P(dg), P(db))
    # dz is overwritten channel by channel only after that channel's sums are taken
    np.testing.assert_array_equal(gbuf, bref["dx"])


def test_backward_tie_at_zero_takes_identity_branch():
    """At z = +0 and z = -0 the stored output lies on the identity branch of f
    (f(y) = y for y >= 0), so the activation's backward passes dz unchanged."""
    z = np.array([0.0, -0.0, 1.0, -0.5]).reshape(1, 1, 4)
    dz = np.array([1.0, 2.0, 4.0, 8.0]).reshape(1, 1, 4)
    bw = oracle.backward_i(z, dz, [1.0], [0.0], [1.0], EPS, 0.25)
    assert bw["dbeta"][0] == 1.0 + 2.0 + 4.0 + 0.25 * 8.0
    bw2 = oracle.backward_ii(z, dz, [1.0], [0.0], [1.0], EPS, 0.25)
    assert bw2["dbeta"][0] == bw["dbeta"][0]


# ---------------------------------------------------------------- comparison blocks (Sec. 3.2)


def test_normalize_closed_form():
    """A channel of m values k +- d (half each) has mu = k and sigma^2 = d^2, so
    xhat = +-d/sqrt(d^2 + eps) exactly (Eq. 1)."""
    d, k, eps = 0.75, 3.0, 0.25
    x = np.array([k + d, k - d] * 4, dtype=np.float64).reshape(2, 1, 4)
    xh = oracle.normalize(x, [k], [d * d], eps)
    expect = np.where(x > k, 1.0, -1.0) * d / np.sqrt(d * d + eps)
    np.testing.assert_array_equal(xh, expect)


def test_normalize_invariants():
    """With the batch statistics, per channel sum xhat = 0 and
    (1/m) sum xhat^2 = sigma^2/(sigma^2 + eps)."""
    x, _, _, _ = _random_layer(3, 7, 33, seed=51)
    eps = 0.1
    mean, var = oracle.batch_stats(x)
    xh = oracle.normalize(x, mean, var, eps)
    m = 3 * 33
    np.testing.assert_allclose(xh.sum(axis=(0, 2)), 0.0, atol=1e-12)
    np.testing.assert_allclose((xh ** 2).sum(axis=(0, 2)) / m, var / (var + eps), rtol=1e-12)


def test_scale_shift_act_equals_forward_z():
    """f(gamma*xhat + beta) on xhat of the batch statistics is the training
    forward's z (Algorithm 1); with dyadic gamma, beta, slope it is exact."""
    x, _, g, b = _random_layer(2, 5, 24, seed=52, gamma_sign=True)
    C = 5
    fw = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    xh = oracle.normalize(x, fw["mean"], fw["var"], EPS)
    z = oracle.scale_shift_act(xh, g, b, SLOPE)
    assert _rel(z, fw["z"]) < 1e-14
    xh2 = np.array([-2.0, -0.5, 0.0, 0.25, 3.0]).reshape(1, 1, 5)
    z2 = oracle.scale_shift_act(xh2, [2.0], [-0.5], 0.25)
    np.testing.assert_array_equal(z2.ravel(), [-1.125, -0.375, -0.125, 0.0, 5.5])


def test_backward_from_xhat_finite_differences():
    """The checkpointing backward from the stored xhat is dL/dx (and dL/dgamma,
    dL/dbeta) of L = sum(dz * z(x)) by central differences."""
    x, dz, g, b = _fd_inputs(100)
    C = x.shape[1]
    fw = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    xh = oracle.normalize(x, fw["mean"], fw["var"], EPS)
    bw = oracle.backward_from_xhat(xh, dz, g, b, fw["var"], EPS, SLOPE)
    h = 1e-6
    fd = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        xp = x.copy()
        xp[idx] += h
        xm = x.copy()
        xm[idx] -= h
        fd[idx] = (_loss(xp, dz, g, b, EPS, SLOPE) - _loss(xm, dz, g, b, EPS, SLOPE)) / (2 * h)
    assert _rel(bw["dx"], fd) < 1e-6
    fdg = np.zeros(C)
    fdb = np.zeros(C)
    for c in range(C):
        e = np.zeros(C)
        e[c] = h
        fdg[c] = (_loss(x, dz, g + e, b, EPS, SLOPE) - _loss(x, dz, g - e, b, EPS, SLOPE)) / (2 * h)
        fdb[c] = (_loss(x, dz, g, b + e, EPS, SLOPE) - _loss(x, dz, g, b - e, EPS, SLOPE)) / (2 * h)
    assert _rel(bw["dgamma"], fdg) < 1e-6
    assert _rel(bw["dbeta"], fdb) < 1e-6


@pytest.mark.parametrize("shape,seed,gsign", [((2, 16, 64), 61, False), ((4, 9, 49), 62, True)])
def test_comparison_backwards_agree(shape, seed, gsign):
    """The standard backward with f' from the stored z, and the checkpointing
    backward from xhat, are the InPlace-ABN gradient (Sec. 3.2: the blocks
    differ in what they store, not in what they compute)."""
    x, dz, g, b = _random_layer(*shape, seed=seed, gamma_sign=gsign)
    C = shape[1]
    fw = oracle.forward_train(x, g, b, np.zeros(C), np.ones(C), EPS, 0.1, SLOPE)
    ref = oracle.backward_i(fw["z"], dz, g, b, fw["var"], EPS, SLOPE)
    st = oracle.backward_standard(x, dz, g, b, fw["mean"], fw["var"], EPS, SLOPE, z=fw["z"])
    xh = oracle.normalize(x, fw["mean"], fw["var"], EPS)
    ck = oracle.backward_from_xhat(xh, dz, g, b, fw["var"], EPS, SLOPE)
    for k in ("dx", "dgamma", "dbeta"):
        assert _rel(st[k], ref[k]) < 1e-11, k
        assert _rel(ck[k], ref[k]) < 1e-11, k


def test_standard_backward_takes_the_sign_of_the_stored_z():
    """Given z, the standard backward's activation derivative follows z (the
    block stores z for exactly that), not the recomputed y: a z whose sign
    disagrees with y changes dbeta by (1 - a) dz at that element."""
    x = np.array([-1.0, 1.0, -3.0, 3.0]).reshape(1, 1, 4)
    dz = np.array([1.0, 2.0, 4.0, 8.0]).reshape(1, 1, 4)
    mean, var = oracle.batch_stats(x)
    a = 0.25
    z_true = np.array([-0.25, 1.0, -0.75, 3.0]).reshape(1, 1, 4)  # signs of y for gamma=1, beta=0
    z_flip = z_true.copy()
    z_flip[0, 0, 0] = 0.0
    by_y = oracle.backward_standard(x, dz, [1.0], [0.0], mean, var, EPS, a)
    by_z = oracle.backward_standard(x, dz, [1.0], [0.0], mean, var, EPS, a, z=z_true)
    flip = oracle.backward_standard(x, dz, [1.0], [0.0], mean, var, EPS, a, z=z_flip)
    assert by_z["dbeta"][0] == by_y["dbeta"][0] == a * 1.0 + 2.0 + a * 4.0 + 8.0
    assert flip["dbeta"][0] == by_z["dbeta"][0] + (1.0 - a) * 1.0


def test_backward_from_xhat_sign_is_exact():
    """The checkpointing backward decides f' on y = gamma*xhat + beta; for
    values where gamma*xhat + beta is exactly 0 it takes the identity branch,
    and the sign of a tiny nonzero y is kept."""
    xh = np.array([0.5, 0.5 + 2.0 ** -40, 0.5 - 2.0 ** -40]).reshape(1, 1, 3)
    dz = np.array([1.0, 2.0, 4.0]).reshape(1, 1, 3)
    bw = oracle.backward_from_xhat(xh, dz, [2.0], [-1.0], [1.0], EPS, 0.25)
    assert bw["dbeta"][0] == 1.0 + 2.0 + 0.25 * 4.0

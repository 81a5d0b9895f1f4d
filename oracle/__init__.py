"""Double-precision CPU oracle for In-Place Activated BatchNorm (arXiv:1712.02616).

TEST INFRASTRUCTURE ONLY.  The oracle is the plain definition of what the GPU
library computes, written from the paper (Sec. 3.1 batch normalisation, Sec. 3.3
leaky ReLU and the BN backward passes, Algorithms 1 and 2, the Appendix) in
plain C with double arithmetic (``iabn_oracle.c``).  Only ``tests/``, the
smoke check and the benchmark's CPU-baseline leg may import this package; the
product library never uses it, and it shares no code with the GPU path.

Arrays are numpy ``float64`` of shape ``(N, C, HW)`` (NCHW with H*W flattened)
or ``(C,)`` for per-channel quantities.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "iabn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_iabn.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile ``iabn_oracle.c`` into ``liboracle_iabn.so`` with gcc (OpenMP)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-fno-fast-math", "-ffp-contract=off", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # Another build of the same source (the sanitizer build of the tests),
    # loaded instead of the default library when named.
    path = os.environ.get("IABN_ORACLE_LIB")
    if not path:
        build(force=False)
        path = _LIB
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(ctypes.c_double)
    I = ctypes.c_int64
    D = ctypes.c_double
    lib.oracle_leaky_relu.argtypes = [D, D]
    lib.oracle_leaky_relu.restype = D
    lib.oracle_leaky_relu_inv.argtypes = [D, D]
    lib.oracle_leaky_relu_inv.restype = D
    lib.oracle_batch_stats.argtypes = [P, I, I, I, P, P]
    lib.oracle_batch_stats.restype = None
    lib.oracle_forward_train.argtypes = [P, I, I, I, P, P, D, D, D, P, P, P, P, P]
    lib.oracle_forward_train.restype = None
    lib.oracle_forward_eval.argtypes = [P, I, I, I, P, P, P, P, D, D, P]
    lib.oracle_forward_eval.restype = None
    for name in ("oracle_backward_i", "oracle_backward_ii"):
        fn = getattr(lib, name)
        fn.argtypes = [P, P, I, I, I, P, P, P, D, D, P, P, P]
        fn.restype = None
    lib.oracle_backward_standard.argtypes = [P, P, P, I, I, I, P, P, P, P, D, D, P, P, P]
    lib.oracle_backward_standard.restype = None
    lib.oracle_normalize.argtypes = [P, I, I, I, P, P, D, P]
    lib.oracle_normalize.restype = None
    lib.oracle_scale_shift_act.argtypes = [P, I, I, I, P, P, D, P]
    lib.oracle_scale_shift_act.restype = None
    lib.oracle_backward_from_xhat.argtypes = [P, P, I, I, I, P, P, P, D, D, P, P, P]
    lib.oracle_backward_from_xhat.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _shape(x: np.ndarray):
    if x.ndim != 3:
        raise ValueError("expected an (N, C, HW) array, got shape %r" % (x.shape,))
    return x.shape


def leaky_relu(y: float, slope: float) -> float:
    """f(y) of Sec. 3.3."""
    return _load().oracle_leaky_relu(float(y), float(slope))


def leaky_relu_inv(z: float, slope: float) -> float:
    """f^-1(z) of Sec. 3.3."""
    return _load().oracle_leaky_relu_inv(float(z), float(slope))


def batch_stats(x):
    """Per-channel mean and biased variance (Sec. 3.1)."""
    x = _f64(x)
    N, C, HW = _shape(x)
    mean = np.empty(C)
    var = np.empty(C)
    _load().oracle_batch_stats(_ptr(x), N, C, HW, _ptr(mean), _ptr(var))
    return mean, var


def forward_train(x, gamma, beta, running_mean, running_var, eps, momentum, slope):
    """Algorithm 1 with the running-statistics update.

    Returns ``dict(z, mean, var, running_mean, running_var)``; the inputs are
    not modified.
    """
    x = _f64(x)
    N, C, HW = _shape(x)
    g, b = _f64(gamma), _f64(beta)
    rm, rv = _f64(running_mean).copy(), _f64(running_var).copy()
    z = np.empty_like(x)
    mean = np.empty(C)
    var = np.empty(C)
    _load().oracle_forward_train(_ptr(x), N, C, HW, _ptr(g), _ptr(b), float(eps), float(momentum),
                                 float(slope), _ptr(rm), _ptr(rv), _ptr(z), _ptr(mean), _ptr(var))
    return dict(z=z, mean=mean, var=var, running_mean=rm, running_var=rv)


def forward_eval(x, gamma, beta, running_mean, running_var, eps, slope):
    """Inference forward with fixed statistics (Sec. 3.1)."""
    x = _f64(x)
    N, C, HW = _shape(x)
    z = np.empty_like(x)
    _load().oracle_forward_eval(_ptr(x), N, C, HW, _ptr(_f64(gamma)), _ptr(_f64(beta)),
                                _ptr(_f64(running_mean)), _ptr(_f64(running_var)), float(eps),
                                float(slope), _ptr(z))
    return z


def _backward_from_z(fn, z, dz, gamma, beta, var, eps, slope):
    z, dz = _f64(z), _f64(dz)
    N, C, HW = _shape(z)
    if dz.shape != z.shape:
        raise ValueError("z and dz shapes differ")
    dx = np.empty_like(z)
    dg = np.empty(C)
    db = np.empty(C)
    fn(_ptr(z), _ptr(dz), N, C, HW, _ptr(_f64(gamma)), _ptr(_f64(beta)), _ptr(_f64(var)),
       float(eps), float(slope), _ptr(dx), _ptr(dg), _ptr(db))
    return dict(dx=dx, dgamma=dg, dbeta=db)


def backward_i(z, dz, gamma, beta, var, eps, slope):
    """Algorithm 2, InPlace-ABN I: gradients from the stored z and sigma^2."""
    return _backward_from_z(_load().oracle_backward_i, z, dz, gamma, beta, var, eps, slope)


def backward_ii(z, dz, gamma, beta, var, eps, slope):
    """Algorithm 2, InPlace-ABN II: gradients as functions of y (Appendix)."""
    return _backward_from_z(_load().oracle_backward_ii, z, dz, gamma, beta, var, eps, slope)


def backward_standard(x, dz, gamma, beta, mean, var, eps, slope, z=None):
    """Standard BN + activation backward from the stored input x (Sec. 3.2).

    With ``z`` (the block's stored output) the activation's derivative comes
    from the sign of z; otherwise from the recomputed y.
    """
    x, dz = _f64(x), _f64(dz)
    N, C, HW = _shape(x)
    zp = None
    if z is not None:
        z = _f64(z)
        if z.shape != x.shape:
            raise ValueError("x and z shapes differ")
        zp = _ptr(z)
    dx = np.empty_like(x)
    dg = np.empty(C)
    db = np.empty(C)
    _load().oracle_backward_standard(_ptr(x), zp, _ptr(dz), N, C, HW, _ptr(_f64(gamma)),
                                     _ptr(_f64(beta)), _ptr(_f64(mean)), _ptr(_f64(var)),
                                     float(eps), float(slope), _ptr(dx), _ptr(dg), _ptr(db))
    return dict(dx=dx, dgamma=dg, dbeta=db)


def normalize(x, mean, var, eps):
    """xhat = (x - mu)/sqrt(sigma^2 + eps) of Eq. (1), for given statistics."""
    x = _f64(x)
    N, C, HW = _shape(x)
    xh = np.empty_like(x)
    _load().oracle_normalize(_ptr(x), N, C, HW, _ptr(_f64(mean)), _ptr(_f64(var)), float(eps),
                             _ptr(xh))
    return xh


def scale_shift_act(xhat, gamma, beta, slope):
    """z = f(gamma*xhat + beta): the checkpointing's recomputation (Sec. 3.2)."""
    xhat = _f64(xhat)
    N, C, HW = _shape(xhat)
    z = np.empty_like(xhat)
    _load().oracle_scale_shift_act(_ptr(xhat), N, C, HW, _ptr(_f64(gamma)), _ptr(_f64(beta)),
                                   float(slope), _ptr(z))
    return z


def backward_from_xhat(xhat, dz, gamma, beta, var, eps, slope):
    """Backward from the stored xhat (BN* of the proposed checkpointing, Sec. 3.2)."""
    return _backward_from_z(_load().oracle_backward_from_xhat, xhat, dz, gamma, beta, var, eps,
                            slope)


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use in this process."""
    return int(_load().oracle_num_threads())

"""Python binding of libiabn: InPlace-ABN (arXiv:1712.02616) on MI355X.

Argument marshalling only.  Every function here has the name and the meaning
of the C entry point declared in ``include/iabn.h``: it checks that the torch
tensors have the layout the library expects, passes raw device pointers, the
shape and the current HIP stream, and turns a nonzero status into
``IabnError``.  All arithmetic happens in the HIP kernels of ``libiabn.so``;
there is no other code path, and calls fail if the library cannot be loaded.

Tensors: activations/gradients are contiguous NCHW (any number of trailing
spatial dims, flattened to HW) in float32, float16 or bfloat16 on a HIP
device; per-channel tensors are contiguous float32 of length C on the same
device.  Calls are asynchronous on ``stream`` (default: torch's current
stream for the tensor's device).
"""

from __future__ import annotations

import ctypes
import math
import threading

import torch

from . import build as _build

__all__ = [
    "IabnError", "load", "library_path", "iabn_version", "iabn_status_string",
    "iabn_workspace_size", "iabn_forward_train", "iabn_forward_eval", "iabn_backward",
    "iabn_forward_stats", "iabn_forward_apply", "iabn_backward_reduce", "iabn_backward_apply",
    "iabn_backward_ii", "iabn_std_forward_train", "iabn_std_backward", "iabn_ckpt_forward_train",
    "iabn_ckpt_recompute", "iabn_ckpt_backward", "iabn_plan", "iabn_forward_train_noalloc",
    "DTYPE_CODES", "OPS",
]

DTYPE_CODES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}

# iabn_op_t: the entry points iabn_plan describes.
OPS = {"forward_train": 0, "backward": 1, "std_forward": 2, "std_backward": 3,
       "ckpt_forward": 4, "ckpt_backward": 5, "forward_eval": 6, "ckpt_recompute": 7}


class _Plan(ctypes.Structure):
    """iabn_plan_t."""
    _fields_ = [("channel_resident", ctypes.c_int), ("access_bytes", ctypes.c_int),
                ("threads", ctypes.c_int), ("reg_accesses", ctypes.c_int),
                ("lds_accesses", ctypes.c_int), ("strips", ctypes.c_int),
                ("xcd_order", ctypes.c_int), ("blocks", ctypes.c_int64),
                ("channels_per_block", ctypes.c_int)]

_lib = None
_lib_lock = threading.Lock()


class IabnError(RuntimeError):
    """A libiabn entry point returned a nonzero status."""

    def __init__(self, fn: str, status: int, detail: str):
        self.status = status
        super().__init__("%s failed with status %d: %s" % (fn, status, detail))


def library_path() -> str:
    return _build.LIB


def load():
    """Load libiabn.so (building it first if it has never been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lib_lock:
        if _lib is None:
            if not _build.is_built():
                _build.build()
            _lib = declare(ctypes.CDLL(_build.LIB))
    return _lib


def declare(lib):
    """Attach the C signatures of include/iabn.h to a loaded libiabn handle."""
    vp, i64, f32, sz, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t, ctypes.c_int
    sig = {
        "iabn_version": ([], i32),
        "iabn_status_string": ([i32], ctypes.c_char_p),
        "iabn_last_error": ([], ctypes.c_char_p),
        "iabn_workspace_size": ([i64, i64, i64, i32], sz),
        "iabn_forward_train": ([vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_forward_train_noalloc": ([vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, f32, i64, i64, i64, vp], i32),
        "iabn_forward_eval": ([vp, i32, vp, vp, vp, vp, f32, f32, i64, i64, i64, vp], i32),
        "iabn_backward": ([vp, vp, i32, vp, vp, vp, vp, vp, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_forward_stats": ([vp, i32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_forward_apply": ([vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_backward_reduce": ([vp, vp, i32, vp, vp, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_backward_apply": ([vp, vp, i32, vp, vp, vp, vp, vp, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_backward_ii": ([vp, vp, i32, vp, vp, vp, vp, vp, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_std_forward_train": ([vp, vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_std_backward": ([vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_ckpt_forward_train": ([vp, vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_ckpt_recompute": ([vp, vp, i32, vp, vp, f32, i64, i64, i64, vp], i32),
        "iabn_ckpt_backward": ([vp, vp, i32, vp, vp, vp, vp, vp, f32, f32, i64, i64, i64, vp, sz, vp], i32),
        "iabn_plan": ([i32, i32, i64, i64, i64, ctypes.POINTER(_Plan)], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


def _check(name: str, rc: int) -> None:
    if rc != 0:
        lib = load()
        raise IabnError(name, rc, (lib.iabn_last_error() or b"").decode() or
                        lib.iabn_status_string(rc).decode())


def _nchw(t: torch.Tensor, what: str):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % what)
    if t.dim() < 2:
        raise ValueError("%s must have at least two dims (N, C, ...), got %r" % (what, tuple(t.shape)))
    if t.dtype not in DTYPE_CODES:
        raise ValueError("%s has unsupported dtype %s" % (what, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous NCHW" % what)
    if t.device.type != "cuda":
        raise ValueError("%s must be on a HIP device" % what)
    N, C = t.shape[0], t.shape[1]
    HW = math.prod(t.shape[2:]) if t.dim() > 2 else 1
    return N, C, HW


def _chan(t, C: int, device, what: str):
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError("%s must be a contiguous float32 tensor" % what)
    if t.numel() != C or t.device != device:
        raise ValueError("%s must hold C=%d values on %s" % (what, C, device))
    return ctypes.c_void_p(t.data_ptr())


def _ptr(t: torch.Tensor):
    return ctypes.c_void_p(t.data_ptr())


def _stream(device, stream):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _workspace(N, C, HW, code, device, workspace, stream=None):
    """The caller's workspace, or a new one from torch's caching allocator.
    A new one is released when this call returns, while the kernels may still
    run: the allocator reuses it only in the order of the stream it was
    recorded on, so it is recorded on the stream the kernels run on."""
    need = iabn_workspace_size(N, C, HW, code)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        if stream is not None:
            if not isinstance(stream, torch.cuda.Stream):
                stream = torch.cuda.ExternalStream(int(stream), device=device)
            workspace.record_stream(stream)
    if workspace.device != device or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor on %s" % device)
    return workspace, ctypes.c_void_p(workspace.data_ptr()), workspace.numel() * workspace.element_size()


def iabn_version() -> int:
    return int(load().iabn_version())


def iabn_status_string(status: int) -> str:
    return load().iabn_status_string(int(status)).decode()


def iabn_workspace_size(N: int, C: int, HW: int, dtype) -> int:
    """Workspace bytes for a shape; ``dtype`` is a torch dtype or a dtype code."""
    code = DTYPE_CODES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return int(load().iabn_workspace_size(int(N), int(C), int(HW), code))


def iabn_plan(op, dtype, N: int, C: int, HW: int) -> dict:
    """How entry point ``op`` (a name of ``OPS`` or an iabn_op_t code) runs a
    shape with aligned tensors: the fields of iabn_plan_t as a dict.  Host
    only."""
    code = DTYPE_CODES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    opc = OPS[op] if isinstance(op, str) else int(op)
    plan = _Plan()
    rc = load().iabn_plan(opc, code, int(N), int(C), int(HW), ctypes.byref(plan))
    _check("iabn_plan", rc)
    return {name: int(getattr(plan, name)) for name, _ in _Plan._fields_}


def iabn_forward_train(x_z, gamma, beta, running_mean, running_var, save_mean, save_var,
                       eps=1e-5, momentum=0.1, slope=0.01, workspace=None, stream=None):
    """Training forward (Algorithm 1), in place over ``x_z``; returns ``x_z``."""
    N, C, HW = _nchw(x_z, "x_z")
    code = DTYPE_CODES[x_z.dtype]
    dev = x_z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (running_mean, "running_mean"), (running_var, "running_var"),
            (save_mean, "save_mean"), (save_var, "save_var"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_forward_train(_ptr(x_z), code, *args, float(eps), float(momentum),
                                   float(slope), N, C, HW, wp, wb, _stream(dev, stream))
    _check("iabn_forward_train", rc)
    return x_z


def iabn_forward_train_noalloc(x_z, gamma, beta, running_mean, running_var, save_mean, save_var,
                               eps=1e-5, momentum=0.1, slope=0.01, stream=None):
    """iabn_forward_train with the library's static scratch in place of a
    workspace (no allocation, here or in the library); returns ``x_z``."""
    N, C, HW = _nchw(x_z, "x_z")
    code = DTYPE_CODES[x_z.dtype]
    dev = x_z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (running_mean, "running_mean"), (running_var, "running_var"),
            (save_mean, "save_mean"), (save_var, "save_var"))]
    rc = load().iabn_forward_train_noalloc(_ptr(x_z), code, *args, float(eps), float(momentum),
                                           float(slope), N, C, HW, _stream(dev, stream))
    _check("iabn_forward_train_noalloc", rc)
    return x_z


def iabn_forward_eval(x_z, gamma, beta, running_mean, running_var, eps=1e-5, slope=0.01,
                      stream=None):
    """Inference forward with the running statistics, in place; returns ``x_z``."""
    N, C, HW = _nchw(x_z, "x_z")
    code = DTYPE_CODES[x_z.dtype]
    dev = x_z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (running_mean, "running_mean"), (running_var, "running_var"))]
    rc = load().iabn_forward_eval(_ptr(x_z), code, *args, float(eps), float(slope), N, C, HW,
                                  _stream(dev, stream))
    _check("iabn_forward_eval", rc)
    return x_z


def iabn_backward(z, dz_dx, gamma, beta, save_var, dgamma, dbeta, eps=1e-5, slope=0.01,
                  workspace=None, stream=None):
    """Backward (Algorithm 2, InPlace-ABN I), in place over ``dz_dx``; returns ``dz_dx``."""
    N, C, HW = _nchw(z, "z")
    if _nchw(dz_dx, "dz_dx") != (N, C, HW) or dz_dx.dtype != z.dtype or dz_dx.device != z.device:
        raise ValueError("dz_dx must match z in shape, dtype and device")
    code = DTYPE_CODES[z.dtype]
    dev = z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (save_var, "save_var"), (dgamma, "dgamma"), (dbeta, "dbeta"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_backward(_ptr(z), _ptr(dz_dx), code, *args, float(eps), float(slope), N, C, HW,
                              wp, wb, _stream(dev, stream))
    _check("iabn_backward", rc)
    return dz_dx


def _same(a, b, what_a, what_b):
    shape = _nchw(a, what_a)
    if _nchw(b, what_b) != shape or b.dtype != a.dtype or b.device != a.device:
        raise ValueError("%s must match %s in shape, dtype and device" % (what_b, what_a))
    return shape


def iabn_backward_ii(z, dz_dx, gamma, beta, save_var, dgamma, dbeta, eps=1e-5, slope=0.01,
                     workspace=None, stream=None):
    """Backward with InPlace-ABN II (gradients in terms of y), in place over ``dz_dx``."""
    N, C, HW = _same(z, dz_dx, "z", "dz_dx")
    code = DTYPE_CODES[z.dtype]
    dev = z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (save_var, "save_var"), (dgamma, "dgamma"), (dbeta, "dbeta"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_backward_ii(_ptr(z), _ptr(dz_dx), code, *args, float(eps), float(slope), N, C,
                                 HW, wp, wb, _stream(dev, stream))
    _check("iabn_backward_ii", rc)
    return dz_dx


def iabn_std_forward_train(x, z, gamma, beta, running_mean, running_var, save_mean, save_var,
                           eps=1e-5, momentum=0.1, slope=0.01, workspace=None, stream=None):
    """Standard block forward: ``x`` kept, ``z`` written; returns ``z``."""
    N, C, HW = _same(x, z, "x", "z")
    code = DTYPE_CODES[x.dtype]
    dev = x.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (running_mean, "running_mean"), (running_var, "running_var"),
            (save_mean, "save_mean"), (save_var, "save_var"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_std_forward_train(_ptr(x), _ptr(z), code, *args, float(eps), float(momentum),
                                       float(slope), N, C, HW, wp, wb, _stream(dev, stream))
    _check("iabn_std_forward_train", rc)
    return z


def iabn_std_backward(x, z, dz_dx, gamma, beta, save_mean, save_var, dgamma, dbeta, eps=1e-5,
                      slope=0.01, workspace=None, stream=None):
    """Standard block backward from ``x`` (and the signs of ``z``), in place over ``dz_dx``."""
    N, C, HW = _same(x, z, "x", "z")
    _same(x, dz_dx, "x", "dz_dx")
    code = DTYPE_CODES[x.dtype]
    dev = x.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (save_mean, "save_mean"), (save_var, "save_var"), (dgamma, "dgamma"), (dbeta, "dbeta"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_std_backward(_ptr(x), _ptr(z), _ptr(dz_dx), code, *args, float(eps),
                                  float(slope), N, C, HW, wp, wb, _stream(dev, stream))
    _check("iabn_std_backward", rc)
    return dz_dx


def iabn_ckpt_forward_train(x_xhat, z, gamma, beta, running_mean, running_var, save_mean,
                            save_var, eps=1e-5, momentum=0.1, slope=0.01, workspace=None,
                            stream=None):
    """Checkpointing forward: xhat over ``x_xhat``, ``z`` written; returns ``z``."""
    N, C, HW = _same(x_xhat, z, "x_xhat", "z")
    code = DTYPE_CODES[x_xhat.dtype]
    dev = x_xhat.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (running_mean, "running_mean"), (running_var, "running_var"),
            (save_mean, "save_mean"), (save_var, "save_var"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_ckpt_forward_train(_ptr(x_xhat), _ptr(z), code, *args, float(eps),
                                        float(momentum), float(slope), N, C, HW, wp, wb,
                                        _stream(dev, stream))
    _check("iabn_ckpt_forward_train", rc)
    return z


def iabn_ckpt_recompute(xhat, z, gamma, beta, slope=0.01, stream=None):
    """z = f(gamma*xhat + beta) from the stored xhat; returns ``z``."""
    N, C, HW = _same(xhat, z, "xhat", "z")
    code = DTYPE_CODES[xhat.dtype]
    dev = xhat.device
    g = _chan(gamma, C, dev, "gamma")
    b = _chan(beta, C, dev, "beta")
    rc = load().iabn_ckpt_recompute(_ptr(xhat), _ptr(z), code, g, b, float(slope), N, C, HW,
                                    _stream(dev, stream))
    _check("iabn_ckpt_recompute", rc)
    return z


def iabn_ckpt_backward(xhat, dz_dx, gamma, beta, save_var, dgamma, dbeta, eps=1e-5, slope=0.01,
                       workspace=None, stream=None):
    """Checkpointing backward from the stored xhat, in place over ``dz_dx``."""
    N, C, HW = _same(xhat, dz_dx, "xhat", "dz_dx")
    code = DTYPE_CODES[xhat.dtype]
    dev = xhat.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (save_var, "save_var"), (dgamma, "dgamma"), (dbeta, "dbeta"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_ckpt_backward(_ptr(xhat), _ptr(dz_dx), code, *args, float(eps), float(slope),
                                   N, C, HW, wp, wb, _stream(dev, stream))
    _check("iabn_ckpt_backward", rc)
    return dz_dx


def iabn_forward_stats(x, workspace, stream=None):
    """First phase of the training forward: partial statistics into ``workspace``."""
    N, C, HW = _nchw(x, "x")
    code = DTYPE_CODES[x.dtype]
    ws, wp, wb = _workspace(N, C, HW, code, x.device, workspace, stream)
    rc = load().iabn_forward_stats(_ptr(x), code, N, C, HW, wp, wb, _stream(x.device, stream))
    _check("iabn_forward_stats", rc)


def iabn_forward_apply(x_z, gamma, beta, running_mean, running_var, save_mean, save_var,
                       eps, momentum, slope, workspace, stream=None):
    """Second phase of the training forward; returns ``x_z``."""
    N, C, HW = _nchw(x_z, "x_z")
    code = DTYPE_CODES[x_z.dtype]
    dev = x_z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (running_mean, "running_mean"), (running_var, "running_var"),
            (save_mean, "save_mean"), (save_var, "save_var"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_forward_apply(_ptr(x_z), code, *args, float(eps), float(momentum),
                                   float(slope), N, C, HW, wp, wb, _stream(dev, stream))
    _check("iabn_forward_apply", rc)
    return x_z


def iabn_backward_reduce(z, dz, gamma, beta, slope, workspace, stream=None):
    """First phase of the backward: partial sums of dy and dy*xhat into ``workspace``."""
    N, C, HW = _nchw(z, "z")
    if _nchw(dz, "dz") != (N, C, HW) or dz.dtype != z.dtype or dz.device != z.device:
        raise ValueError("dz must match z in shape, dtype and device")
    code = DTYPE_CODES[z.dtype]
    dev = z.device
    g = _chan(gamma, C, dev, "gamma")
    b = _chan(beta, C, dev, "beta")
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_backward_reduce(_ptr(z), _ptr(dz), code, g, b, float(slope), N, C, HW, wp, wb,
                                     _stream(dev, stream))
    _check("iabn_backward_reduce", rc)


def iabn_backward_apply(z, dz_dx, gamma, beta, save_var, dgamma, dbeta, eps, slope, workspace,
                        stream=None):
    """Second phase of the backward; returns ``dz_dx``."""
    N, C, HW = _nchw(z, "z")
    if _nchw(dz_dx, "dz_dx") != (N, C, HW) or dz_dx.dtype != z.dtype or dz_dx.device != z.device:
        raise ValueError("dz_dx must match z in shape, dtype and device")
    code = DTYPE_CODES[z.dtype]
    dev = z.device
    args = [_chan(t, C, dev, n) for t, n in ((gamma, "gamma"), (beta, "beta"),
            (save_var, "save_var"), (dgamma, "dgamma"), (dbeta, "dbeta"))]
    ws, wp, wb = _workspace(N, C, HW, code, dev, workspace, stream)
    rc = load().iabn_backward_apply(_ptr(z), _ptr(dz_dx), code, *args, float(eps), float(slope),
                                    N, C, HW, wp, wb, _stream(dev, stream))
    _check("iabn_backward_apply", rc)
    return dz_dx

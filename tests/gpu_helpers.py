"""Shared helpers of the GPU parity tests (not a test module)."""

from __future__ import annotations

import numpy as np
import torch

import paper_1712_02616_amd as iabn
import workloads

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

# Gates on the max relative error (floored, see max_rel): fp32 storage 1e-4,
# fp16/bf16 storage with fp32 arithmetic 2e-2.
TOL = {"f32": 1e-4, "f16": 2e-2, "bf16": 2e-2}


def say(msg: str) -> None:
    print(msg, flush=True)


def to_device(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Storage-format numpy array (bf16 as uint16 bits) -> device tensor."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> exact float64 numpy array."""
    return t.detach().to("cpu").to(torch.float64).numpy()


def max_rel(got: np.ndarray, ref: np.ndarray, floor_frac: float = 1e-3,
            floor_abs: float = 0.0) -> float:
    """max_i |got_i - ref_i| / max(|ref_i|, floor_frac * max_j |ref_j|, floor_abs)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    scale = np.max(np.abs(ref))
    denom = np.maximum(np.maximum(np.abs(ref), floor_frac * scale), floor_abs)
    denom = np.where(denom > 0, denom, 1.0)
    return float(np.max(np.abs(got - ref) / denom))


def assert_close(name: str, got, ref, dtype: str, mask=None, floor_abs: float = 0.0) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "%s has non-finite values" % name
    if mask is not None:
        err = max_rel(got[mask], ref[mask], floor_abs=floor_abs) if mask.any() else 0.0
    else:
        err = max_rel(got, ref, floor_abs=floor_abs)
    tol = TOL[dtype]
    assert err <= tol, "%s: max rel err %.3e > %.1e (%s)" % (name, err, tol, dtype)
    return err


class GpuLayer:
    """A layer's inputs on the device plus the per-channel buffers."""

    def __init__(self, inp: workloads.LayerInputs, device="cuda"):
        self.inp = inp
        self.dtype = inp.dtype
        N, C, HW = inp.x.shape
        self.shape = (N, C, HW)
        self.x = to_device(inp.x, inp.dtype, device)
        self.dz = to_device(inp.dz, inp.dtype, device)
        self.gamma = torch.from_numpy(inp.gamma).to(device)
        self.beta = torch.from_numpy(inp.beta).to(device)
        self.running_mean = torch.from_numpy(inp.running_mean.copy()).to(device)
        self.running_var = torch.from_numpy(inp.running_var.copy()).to(device)
        self.save_mean = torch.empty(C, dtype=torch.float32, device=device)
        self.save_var = torch.empty(C, dtype=torch.float32, device=device)
        self.dgamma = torch.empty(C, dtype=torch.float32, device=device)
        self.dbeta = torch.empty(C, dtype=torch.float32, device=device)
        self.workspace = torch.empty(max(iabn.iabn_workspace_size(N, C, HW, TORCH_DTYPES[inp.dtype]), 1),
                                     dtype=torch.uint8, device=device)

    def forward_train(self, eps, momentum, slope, path="entry"):
        """path "entry": iabn_forward_train (which may pick the channel-resident
        kernel); "phases": iabn_forward_stats + iabn_forward_apply."""
        if path == "entry":
            iabn.iabn_forward_train(self.x, self.gamma, self.beta, self.running_mean,
                                    self.running_var, self.save_mean, self.save_var, eps, momentum,
                                    slope, workspace=self.workspace)
        else:
            iabn.iabn_forward_stats(self.x, self.workspace)
            iabn.iabn_forward_apply(self.x, self.gamma, self.beta, self.running_mean,
                                    self.running_var, self.save_mean, self.save_var, eps, momentum,
                                    slope, self.workspace)

    def backward(self, eps, slope, z=None, save_var=None, path="entry"):
        z = self.x if z is None else z
        sv = self.save_var if save_var is None else save_var
        if path == "entry":
            iabn.iabn_backward(z, self.dz, self.gamma, self.beta, sv, self.dgamma, self.dbeta, eps,
                               slope, workspace=self.workspace)
        else:
            iabn.iabn_backward_reduce(z, self.dz, self.gamma, self.beta, slope, self.workspace)
            iabn.iabn_backward_apply(z, self.dz, self.gamma, self.beta, sv, self.dgamma, self.dbeta,
                                     eps, slope, self.workspace)

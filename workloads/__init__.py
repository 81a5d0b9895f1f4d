"""Seeded synthetic inputs for the InPlace-ABN workloads.

This module only draws random numbers and converts them to the storage
formats (fp32, fp16, bf16); it holds none of the method's arithmetic.  Both the
oracle-side tests and the GPU-side tests and benchmark take their inputs from
here, so the two sides see bit-identical storage values.

Recipe (per layer of a workload, all draws in float64 from numpy's PCG64):
  mu_c ~ U(-2, 2), sigma_c ~ U(0.5, 3)              per channel
  gamma_c ~ U(0.5, 1.5)  (times a random sign when ``gamma_sign``)
  beta_c ~ N(0, 0.1^2)
  x[n, c, :] = mu_c + sigma_c * N(0, 1)
  dz[n, c, :] = dz_std * N(0, 1)
then x and dz are rounded to the storage type with round-to-nearest-even
(bf16 goes through float32, also round-to-nearest-even).  Parameters stay
fp32.  Running statistics start at mean 0, variance 1.

Each (layer, sample n, tensor) slab has its own generator keyed by
``SeedSequence([seed, layer, n, tensor])`` so that slabs can be drawn in
parallel threads and the result does not depend on the thread count.
"""

from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

DTYPES = ("f32", "f16", "bf16")
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2}

SLOPE = 0.01
EPS = 1e-5
MOMENTUM = 0.1
BASE_SEED = 1712


@dataclasses.dataclass(frozen=True)
class Workload:
    index: int
    name: str
    dtype: str
    layers: tuple  # tuple of (N, C, HW)
    dz_std: float
    gamma_sign: bool = False
    slope: float = SLOPE
    eps: float = EPS
    momentum: float = MOMENTUM

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def elements(self) -> int:
        return sum(n * c * hw for n, c, hw in self.layers)

    @property
    def tensor_bytes(self) -> int:
        return self.elements * ELEM_BYTES[self.dtype]


_BACKBONE = (((8, 256, 128 * 128),) * 3 + ((8, 512, 64 * 64),) * 4 +
             ((8, 1024, 64 * 64),) * 23 + ((8, 2048, 64 * 64),) * 3)

WORKLOADS = {
    # Tiny layer, fp32: N=2, C=16, H=W=8, dz ~ N(0, 1).
    1: Workload(1, "tiny_2x16x8x8_f32", "f32", ((2, 16, 64),), dz_std=1.0),
    # ResNet-style layer, fp32: N=32, C=256, H=W=56, dz ~ N(0, 1e-2).
    2: Workload(2, "resnet_32x256x56x56_f32", "f32", ((32, 256, 56 * 56),), dz_std=0.1),
    # Segmentation crop, fp16 storage: N=4, C=256, H=W=192, gamma with random sign.
    3: Workload(3, "segcrop_4x256x192x192_f16", "f16", ((4, 256, 192 * 192),), dz_std=0.1,
                gamma_sign=True),
    # Wide-channel deep layer, bf16 storage: N=16, C=2048, H=W=28, dz ~ N(0, 1).
    4: Workload(4, "wide_16x2048x28x28_bf16", "bf16", ((16, 2048, 28 * 28),), dz_std=1.0),
    # ResNet-101-like backbone at N=8, 512x512 input, output stride 8: the four
    # BN shape groups (C, H=W) = (256,128), (512,64), (1024,64), (2048,64) with
    # 3, 4, 23, 3 layers, fp16 storage; dz ~ N(0, 1e-2).
    5: Workload(5, "backbone_r101_os8_n8_512px_f16", "f16", _BACKBONE, dz_std=0.1),
}


def single_layer(N: int, C: int, H: int, W: int, dtype: str) -> Workload:
    """A one-layer workload of any shape with the ResNet layer's value
    distributions (dz ~ N(0, 1e-2)) and seed 1712; for measuring layer
    shapes outside the five workloads above."""
    if dtype not in DTYPES:
        raise ValueError("unknown dtype %r" % dtype)
    if min(N, C, H, W) < 1:
        raise ValueError("every size must be positive")
    return Workload(0, "layer_%dx%dx%dx%d_%s" % (N, C, H, W, dtype), dtype, ((N, C, H * W),),
                    dz_std=0.1)


def f64_to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage format (RNE).

    Returns float32 / float16 arrays, or uint16 bit patterns for bf16.
    """
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32)
    if dtype == "f16":
        return np.asarray(a, dtype=np.float16)
    if dtype == "bf16":
        return f32_to_bf16_bits(np.asarray(a, dtype=np.float32))
    raise ValueError("unknown dtype %r" % dtype)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even; NaN stays NaN."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = ((u + rounding) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x0040)).astype(np.uint16)
    return out


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact conversion of storage values to float64."""
    if dtype in ("f32", "f16"):
        return np.asarray(a, dtype=np.float64)
    if dtype == "bf16":
        bits = np.ascontiguousarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError("unknown dtype %r" % dtype)


def storage_numpy_dtype(dtype: str):
    return {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[dtype]


@dataclasses.dataclass
class LayerInputs:
    """One layer's inputs; x and dz are in storage format, shape (N, C, HW)."""
    x: np.ndarray
    dz: np.ndarray
    gamma: np.ndarray  # float32 [C]
    beta: np.ndarray  # float32 [C]
    running_mean: np.ndarray  # float32 [C]
    running_var: np.ndarray  # float32 [C]
    dtype: str

    @property
    def shape(self):
        return self.x.shape


def _rng(*key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def _threads(threads):
    if threads:
        return threads
    return max(1, min(16, os.cpu_count() or 1))


def make_layer(N: int, C: int, HW: int, dtype: str, seed: int, layer: int = 0,
               dz_std: float = 1.0, gamma_sign: bool = False, threads: int = 0) -> LayerInputs:
    """Draw one layer's inputs with the recipe in the module docstring."""
    if dtype not in DTYPES:
        raise ValueError("unknown dtype %r" % dtype)
    prng = _rng(seed, layer)
    mu = prng.uniform(-2.0, 2.0, C)
    sigma = prng.uniform(0.5, 3.0, C)
    gamma = prng.uniform(0.5, 1.5, C)
    if gamma_sign:
        gamma = gamma * np.where(prng.uniform(0.0, 1.0, C) < 0.5, -1.0, 1.0)
    beta = prng.normal(0.0, 0.1, C)

    x = np.empty((N, C, HW), dtype=storage_numpy_dtype(dtype))
    dz = np.empty((N, C, HW), dtype=storage_numpy_dtype(dtype))

    def slab(n):
        g = _rng(seed, layer, n, 0)
        x[n] = f64_to_storage(mu[:, None] + sigma[:, None] * g.standard_normal((C, HW)), dtype)
        g = _rng(seed, layer, n, 1)
        dz[n] = f64_to_storage(dz_std * g.standard_normal((C, HW)), dtype)

    if N * C * HW >= (1 << 22) and N > 1:
        with ThreadPoolExecutor(_threads(threads)) as ex:
            list(ex.map(slab, range(N)))
    else:
        for n in range(N):
            slab(n)
    return LayerInputs(x=x, dz=dz, gamma=gamma.astype(np.float32), beta=beta.astype(np.float32),
                       running_mean=np.zeros(C, np.float32), running_var=np.ones(C, np.float32),
                       dtype=dtype)


def workload_layer(w: Workload, layer: int, threads: int = 0) -> LayerInputs:
    N, C, HW = w.layers[layer]
    return make_layer(N, C, HW, w.dtype, w.seed, layer, dz_std=w.dz_std,
                      gamma_sign=w.gamma_sign, threads=threads)


def make_layer_device(N: int, C: int, HW: int, dtype: str, seed: int, dz_std: float = 0.1,
                      gamma_sign: bool = False, device="cuda"):
    """One layer drawn directly on the device, for tensors too large to build
    on the host: the per-channel parameters follow the module recipe (numpy,
    ``SeedSequence([seed, 0])``); x and dz are drawn channel by channel with
    torch's seeded device generator (Philox) in float32 and rounded to the
    storage type (round to nearest even).  Same distributions as
    ``make_layer``, a different stream of numbers.

    Returns ``(x, dz, params)``: device tensors of shape (N, C, HW) in the
    storage type and a ``LayerInputs`` whose x/dz are None.
    """
    import torch

    if dtype not in DTYPES:
        raise ValueError("unknown dtype %r" % dtype)
    prng = _rng(seed, 0)
    mu = prng.uniform(-2.0, 2.0, C)
    sigma = prng.uniform(0.5, 3.0, C)
    gamma = prng.uniform(0.5, 1.5, C)
    if gamma_sign:
        gamma = gamma * np.where(prng.uniform(0.0, 1.0, C) < 0.5, -1.0, 1.0)
    beta = prng.normal(0.0, 0.1, C)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    x = torch.empty((N, C, HW), dtype=tdt, device=device)
    dz = torch.empty((N, C, HW), dtype=tdt, device=device)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    # Channel by channel while channels are large, in groups otherwise.
    step = max(1, (1 << 26) // max(1, N * HW))
    for c0 in range(0, C, step):
        c1 = min(C, c0 + step)
        mu_t = torch.tensor(mu[c0:c1], dtype=torch.float32, device=device)[None, :, None]
        sd_t = torch.tensor(sigma[c0:c1], dtype=torch.float32, device=device)[None, :, None]
        r = torch.randn((N, c1 - c0, HW), generator=g, device=device, dtype=torch.float32)
        x[:, c0:c1] = (r * sd_t + mu_t).to(tdt)
        r = torch.randn((N, c1 - c0, HW), generator=g, device=device, dtype=torch.float32)
        dz[:, c0:c1] = (r * float(dz_std)).to(tdt)
        del r
    params = LayerInputs(x=None, dz=None, gamma=gamma.astype(np.float32),
                         beta=beta.astype(np.float32), running_mean=np.zeros(C, np.float32),
                         running_var=np.ones(C, np.float32), dtype=dtype)
    return x, dz, params

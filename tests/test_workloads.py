"""The seeded input generator: storage rounding and reproducibility (CPU only)."""

import numpy as np
import pytest
import torch

import workloads


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 7,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 65504.0, 3.4e38, 1e-40],
                                 np.float32)])
    ours = workloads.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = workloads.storage_to_f64(ours, "bf16")
    np.testing.assert_array_equal(back, torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16)
                                  .to(torch.float64).numpy())


def test_f16_rounding_is_numpy_rne():
    a = np.array([1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, -2.5e-8, 70000.0])
    s = workloads.f64_to_storage(a, "f16")
    assert s.dtype == np.float16
    np.testing.assert_array_equal(s.astype(np.float64), [1.0, 1.0 + 2.0 ** -9, -0.0, np.inf])


def test_generation_is_reproducible_and_thread_independent():
    a = workloads.make_layer(4, 8, 70000, "bf16", seed=99, threads=1)
    b = workloads.make_layer(4, 8, 70000, "bf16", seed=99, threads=4)
    np.testing.assert_array_equal(a.x, b.x)
    np.testing.assert_array_equal(a.dz, b.dz)
    np.testing.assert_array_equal(a.gamma, b.gamma)
    c = workloads.make_layer(4, 8, 70000, "bf16", seed=100, threads=4)
    assert not np.array_equal(a.x, c.x)


def test_distribution_recipe():
    inp = workloads.make_layer(2, 64, 4096, "f32", seed=7, dz_std=0.1, gamma_sign=True)
    x = inp.x.astype(np.float64)
    mu = x.mean(axis=(0, 2))
    sd = x.std(axis=(0, 2))
    assert np.all((mu > -2.1) & (mu < 2.1))
    assert np.all((sd > 0.45) & (sd < 3.1))
    assert np.all((np.abs(inp.gamma) >= 0.5) & (np.abs(inp.gamma) <= 1.5))
    assert (inp.gamma < 0).any() and (inp.gamma > 0).any()
    assert abs(inp.dz.std() - 0.1) < 0.005


def test_workload_table():
    w = workloads.WORKLOADS
    assert w[2].elements == 32 * 256 * 3136
    assert w[5].elements == 1140850688
    assert len(w[5].layers) == 33
    assert [w[k].dtype for k in range(1, 6)] == ["f32", "f32", "f16", "bf16", "f16"]


def test_single_layer_workload():
    w = workloads.single_layer(8, 64, 256, 256, "f16")
    assert w.layers == ((8, 64, 65536),) and w.dtype == "f16" and w.seed == workloads.BASE_SEED
    assert w.dz_std == 0.1 and w.name == "layer_8x64x256x256_f16"
    with pytest.raises(ValueError):
        workloads.single_layer(8, 64, 0, 256, "f16")
    with pytest.raises(ValueError):
        workloads.single_layer(8, 64, 16, 16, "f64")

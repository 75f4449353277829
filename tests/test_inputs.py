"""The seeded input generator: bf16 rounding and reproducibility."""
import numpy as np
import torch

from paper_2105_13480_amd import inputs


def test_bf16_rounding_matches_torch():
    """Library pin: torch's float32 -> bfloat16 cast rounds to nearest even."""
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32),
        rng.uniform(-1e30, 1e30, 1000).astype(np.float32),
        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -3.4e38, 1e-40], dtype=np.float32),
    ])
    ours = inputs.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_ties_to_even():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7: ties to the even mantissa (1.0)
    assert inputs.f32_to_bf16_bits(np.float32([1.00390625]))[0] == 0x3F80
    # 1 + 3*2^-8 lies halfway between 1+2^-7 (odd) and 1+2^-6 (even)
    assert inputs.f32_to_bf16_bits(np.float32([1.01171875]))[0] == 0x3F82
    assert inputs.bf16_bits_to_f32(np.uint16([0x3F82]))[0] == np.float32(1.015625)


def test_workloads_reproducible_and_shaped():
    w = inputs.BY_NAME["tiny3x3_f32"]
    a1, k1 = inputs.make_inputs(w)
    a2, k2 = inputs.make_inputs(w)
    assert a1.dtype == np.float32 and a1.shape == (1, 16, 18, 18) and k1.shape == (16, 16, 3, 3)
    assert np.array_equal(a1, a2) and np.array_equal(k1, k2)
    assert a1.min() >= -1 and a1.max() <= 1
    assert w.flops == 2 * 16 * 16 * 9 * 256


def test_workload_extents():
    ext = {w.name: (w.Nx, w.Ny) for w in inputs.WORKLOADS}
    assert ext["tiny3x3_f32"] == (18, 18)
    assert ext["conv3x3_b32"] == (58, 58)
    assert ext["conv3x3_s2_b64"] == (57, 57)
    assert ext["pointwise_b256"] == (14, 14)
    assert ext["stem7x7_s2_b64"] == (229, 229)
    assert ext["pointwise_s2_b64"] == (55, 55)
    assert ext["late3x3_b1"] == (9, 9)


def test_he_normal_scale():
    In, Ker = inputs.make_arrays(1, 64, 256, 2, 2, 3, 3, 1, 1, "f32", seed_in=1, seed_ker=2)
    assert abs(Ker.std() - np.sqrt(2.0 / (64 * 9))) < 0.02 * np.sqrt(2.0 / (64 * 9))

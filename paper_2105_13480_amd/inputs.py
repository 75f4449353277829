"""Seeded synthetic inputs for the CNN forward contraction.

This module holds no convolution arithmetic.  It is the only code shared by
the GPU path's tests/benchmark and the CPU oracle: both read the same arrays.

Every workload is synthetic.  The paper runs no experiments and uses no
dataset; the shapes below are ResNet-style layers (stem, 3x3, strided 3x3,
pointwise) and the value distributions are a uniform activation and a
He-normal kernel, N(0, 2/fan_in) with fan_in = Nc*Nr*Ns (the second
parameter is the variance).

Recipe: numpy PCG64 (``default_rng``) seeded with 1000*i+1 for In and
1000*i+2 for Ker, where i is the 1-based workload number; values are drawn
in float64, rounded to float32, and for bfloat16 workloads rounded once more
to bfloat16 with round-to-nearest-even on the host.  bfloat16 arrays are
returned as uint16 bit patterns so no library rounding is involved.

Layouts are those of the library: In[Nb][Nc][Nx][Ny] with
Nx = sw*(Nw-1)+Nr, Ny = sh*(Nh-1)+Ns; Ker[Nk][Nc][Nr][Ns].
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    index: int          # 1-based workload number (seeds derive from it)
    Nb: int
    Nc: int
    Nk: int
    Nw: int
    Nh: int
    Nr: int
    Ns: int
    sw: int
    sh: int
    dtype: str          # "f32" (fp32 in/out) or "bf16" (bf16 in, fp32 accumulate)
    in_dist: tuple = ("uniform", 0.0, 1.0)
    ker_dist: tuple = ("he",)
    note: str = field(default="", compare=False)

    @property
    def Nx(self) -> int:
        return self.sw * (self.Nw - 1) + self.Nr

    @property
    def Ny(self) -> int:
        return self.sh * (self.Nh - 1) + self.Ns

    @property
    def flops(self) -> int:
        """2 * Nb Nk Nc Nr Ns Nw Nh (one multiply and one add per term)."""
        return 2 * self.Nb * self.Nk * self.Nc * self.Nr * self.Ns * self.Nw * self.Nh

    def dims(self):
        return (self.Nb, self.Nc, self.Nk, self.Nw, self.Nh, self.Nr, self.Ns, self.sw, self.sh)


WORKLOADS = [
    Workload("tiny3x3_f32", 1, 1, 16, 16, 16, 16, 3, 3, 1, 1, "f32",
             ("uniform", -1.0, 1.0), ("uniform", -1.0, 1.0),
             "tiny: Nb=1 Nc=Nk=16, 16x16 out, 3x3, stride 1, fp32"),
    Workload("conv3x3_b32", 2, 32, 64, 64, 56, 56, 3, 3, 1, 1, "bf16",
             ("uniform", 0.0, 1.0), ("he",),
             "3x3 conv: Nb=32 Nc=Nk=64, 56x56 out, stride 1"),
    Workload("conv3x3_s2_b64", 3, 64, 128, 256, 28, 28, 3, 3, 2, 2, "bf16",
             ("uniform", 0.0, 1.0), ("he",),
             "strided 3x3 conv: Nb=64 Nc=128 Nk=256, 28x28 out, stride 2"),
    Workload("pointwise_b256", 4, 256, 1024, 256, 14, 14, 1, 1, 1, 1, "bf16",
             ("uniform", 0.0, 1.0), ("he",),
             "pointwise conv (pure GEMM): Nb=256 Nc=1024 Nk=256, 14x14"),
    Workload("stem7x7_s2_b64", 5, 64, 3, 64, 112, 112, 7, 7, 2, 2, "bf16",
             ("uniform", -1.0, 1.0), ("he",),
             "large-stencil input layer: Nb=64 Nc=3 Nk=64, 112x112 out, 7x7, stride 2"),
    Workload("pointwise_s2_b64", 6, 64, 256, 512, 28, 28, 1, 1, 2, 2, "bf16",
             ("uniform", 0.0, 1.0), ("he",),
             "supplementary strided pointwise: Nb=64 Nc=256 Nk=512, 28x28 out, 1x1, stride 2"),
    Workload("late3x3_b1", 7, 1, 512, 512, 7, 7, 3, 3, 1, 1, "bf16",
             ("uniform", 0.0, 1.0), ("he",),
             "supplementary deep layer at batch 1: Nb=1 Nc=Nk=512, 7x7 out, 3x3, stride 1 "
             "(few output tiles, many channels: the channel-split plans)"),
]

BY_NAME = {w.name: w for w in WORKLOADS}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16.  NaN maps to a quiet NaN.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact float32 values of bfloat16 bit patterns."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw(rng: np.random.Generator, shape, dist, fan_in: int) -> np.ndarray:
    kind = dist[0]
    if kind == "uniform":
        v = rng.uniform(dist[1], dist[2], size=shape)
    elif kind == "he":
        v = rng.standard_normal(size=shape) * np.sqrt(2.0 / fan_in)
    elif kind == "int":
        v = rng.integers(dist[1], dist[2] + 1, size=shape).astype(np.float64)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return v.astype(np.float32)


def make_arrays(Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, dtype, *, seed_in, seed_ker,
                in_dist=("uniform", 0.0, 1.0), ker_dist=("he",)):
    """Seeded (In, Ker) for an arbitrary problem.

    dtype "f32" returns float32 arrays; "bf16" returns uint16 bf16 patterns.
    ``("int", lo, hi)`` draws integers in [lo, hi] (exact in both dtypes).
    """
    Nx = sw * (Nw - 1) + Nr
    Ny = sh * (Nh - 1) + Ns
    fan_in = Nc * Nr * Ns
    In = _draw(np.random.default_rng(seed_in), (Nb, Nc, Nx, Ny), in_dist, fan_in)
    Ker = _draw(np.random.default_rng(seed_ker), (Nk, Nc, Nr, Ns), ker_dist, fan_in)
    if dtype == "bf16":
        return f32_to_bf16_bits(In), f32_to_bf16_bits(Ker)
    if dtype == "f32":
        return In, Ker
    raise ValueError(f"unknown dtype {dtype!r}")


def make_inputs(w: Workload, *, seed_offset: int = 0):
    """(In, Ker) of a named workload with its canonical seeds."""
    return make_arrays(*w.dims(), w.dtype,
                       seed_in=1000 * w.index + 1 + seed_offset,
                       seed_ker=1000 * w.index + 2 + seed_offset,
                       in_dist=w.in_dist, ker_dist=w.ker_dist)

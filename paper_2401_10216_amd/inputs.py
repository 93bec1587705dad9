"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and lays them out; it does none of the
Gaunt-product arithmetic, so both the HIP path and the fp64 oracle can consume
its arrays.  Quantities that need the method's own functions (e.g. the real SH
of an edge direction) are handed over as their raw random ingredients (the
direction and the radial weights) and each side evaluates them itself.

Workloads (the paper ships no data; these stand in for its benchmarks):
  * ``tiny``      : B=1024 pairs, C=1, L1=L2=Lout=2, iid N(0,1).
  * ``edge``      : B=65536 edges, C=128 channels, L=6.  x1 ~ N(0,1); x2 is the
                    real SH of a random unit edge vector (shared by all channels
                    of an edge) times per-(edge, channel, degree) radial weights
                    h ~ N(0,1).  Models the equivariant convolution of Sec. 3.3
                    with the OC20 shape of the paper's experiments (L in {4,6},
                    128 channels).
  * ``manybody``  : 64 molecules x 27 atoms = 1728 nodes, C=256, input L=2,
                    x ~ N(0,1) / sqrt(2l+1) per degree, nu=3, Lout=3 (the 3BPA /
                    MACE shape: L=2, 256 channels, correlation order 3).
  * ``sweep``     : B*C = 262144 vectors ([2048, 128]), L1=L2=Lout=L in
                    {4, 8, 16, 32, 64}, iid N(0,1).
  * ``highdeg``   : B=32768, C=64, L1=L2=Lout=16, inputs rounded to bf16.
  * ``mix``       : channel mixing, B=8192, C1=C2=Co=32, L=6: x1, x2 ~ N(0,1),
                    W ~ N(0, 1/C^2) (the O(C^2)-products combination rule).

Seeds: numpy PCG64 with seed 1000 + workload index (1..6); subsample indices use
seed + 100.
"""
from __future__ import annotations

import numpy as np

WORKLOADS = {
    "tiny": dict(index=1, B=1024, C=1, L1=2, L2=2, Lout=2),
    "edge": dict(index=2, B=65536, C=128, L1=6, L2=6, Lout=6),
    "manybody": dict(index=3, B=1728, C=256, L=2, nu=3, Lout=3),
    "sweep": dict(index=4, B=2048, C=128, Ls=(4, 8, 16, 32, 64)),
    "highdeg": dict(index=5, B=32768, C=64, L1=16, L2=16, Lout=16),
    "mix": dict(index=6, B=8192, C=32, L1=6, L2=6, Lout=6),
}


def nsh(L: int) -> int:
    return (L + 1) * (L + 1)


def rng_for(index: int, offset: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(1000 + index + offset))


def degree_of_index(L: int) -> np.ndarray:
    """Degree l of every coefficient slot i = l*l + l + m, i < (L+1)^2."""
    return np.concatenate([np.full(2 * l + 1, l) for l in range(L + 1)])


def normal(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def round_to_bf16(x: np.ndarray):
    """Round float32 to bfloat16 (nearest, ties to even).

    Returns (bits uint16, values float32) where values are the bf16 numbers
    widened back to float32 exactly.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    bits = (rounded >> np.uint32(16)).astype(np.uint16)
    vals = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return bits, vals


def pair_inputs(index: int, B: int, C: int, L1: int, L2: int):
    """Two iid N(0,1) feature sets x1[B,C,(L1+1)^2], x2[B,C,(L2+1)^2]."""
    rng = rng_for(index)
    x1 = normal(rng, (B, C, nsh(L1)))
    x2 = normal(rng, (B, C, nsh(L2)))
    return x1, x2


def edge_inputs(B: int = 65536, C: int = 128, L: int = 6, index: int = 2):
    """Ingredients of the edge workload.

    Returns x1[B,C,(L+1)^2] ~ N(0,1), unit edge vectors r[B,3] and radial
    weights h[B,C,L+1] ~ N(0,1).  The filter is x2[b,c,(l,m)] = h[b,c,l] *
    Y_l^m(r_b); each side computes it with its own spherical harmonics.
    """
    rng = rng_for(index)
    x1 = normal(rng, (B, C, nsh(L)))
    r = rng.standard_normal(size=(B, 3))
    r /= np.linalg.norm(r, axis=1, keepdims=True)
    h = normal(rng, (B, C, L + 1))
    return x1, r.astype(np.float64), h


def manybody_inputs(N: int = 1728, C: int = 256, L: int = 2, index: int = 3):
    """x[N,C,(L+1)^2] ~ N(0,1) / sqrt(2l+1) for the coefficient's degree l."""
    rng = rng_for(index)
    x = normal(rng, (N, C, nsh(L)))
    scale = (1.0 / np.sqrt(2.0 * degree_of_index(L) + 1.0)).astype(np.float32)
    return x * scale


def sweep_inputs(L: int, B: int = 2048, C: int = 128, index: int = 4):
    """Degree-sweep pair at degree L (seed depends on L so sizes are independent)."""
    rng = np.random.Generator(np.random.PCG64(1000 + index + 10 * L))
    x1 = normal(rng, (B, C, nsh(L)))
    x2 = normal(rng, (B, C, nsh(L)))
    return x1, x2


def highdeg_inputs(B: int = 32768, C: int = 64, L: int = 16, index: int = 5):
    """bf16-rounded N(0,1) pair: returns (bits1, bits2, vals1, vals2)."""
    x1, x2 = pair_inputs(index, B, C, L, L)
    b1, v1 = round_to_bf16(x1)
    b2, v2 = round_to_bf16(x2)
    return b1, b2, v1, v2


def mix_inputs(B: int = 8192, C: int = 32, L: int = 6, index: int = 6):
    """Channel-mixing workload: x1, x2 [B, C, (L+1)^2] ~ N(0,1) and a weight
    tensor W [C, C, C] ~ N(0, 1 / C^2)."""
    rng = rng_for(index)
    x1 = normal(rng, (B, C, nsh(L)))
    x2 = normal(rng, (B, C, nsh(L)))
    W = normal(rng, (C, C, C)) / np.float32(C)
    return x1, x2, W


def output_gradient(index: int, shape) -> np.ndarray:
    """Seeded N(0,1) output gradient dy of a workload (for its backward pass)."""
    return normal(rng_for(index, 200), shape)


def sample_indices(index: int, total: int, count: int) -> np.ndarray:
    """Sorted distinct product indices for subsampled checks."""
    rng = rng_for(index, 100)
    count = min(count, total)
    return np.sort(rng.choice(total, size=count, replace=False))

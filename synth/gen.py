"""Seeded input generator (workload recipe of the decode-linear benchmarks).

Draw order from ``numpy.random.Generator(PCG64(seed))`` is fixed:
X, codes, scales, zero-points, outlier positions, outlier values.

Layouts produced (the library's input format):

* ``X``       uint16 ``[M][K]``        bf16 bit patterns, row-major.
* ``Wq``      uint32 ``[K/8][N]``      code of (k, n) in bits 4*(k%8)..+3 of
                                        word ``Wq[k//8, n]``.
* ``scales``  uint16 ``[K/G][N]``      fp16 bit patterns.
* ``zeros``   uint32 ``[K/G][N/8]``    zero-point of (g, n) in bits
                                        4*(n%8)..+3 of word ``zeros[g, n//8]``.
* outliers    ``k`` int32, ``n`` int32, ``v`` uint16 (bf16 bits), unordered
              COO triples; the INT4 code at every outlier position equals its
              group's zero-point, so the two supports are disjoint.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# Workloads: synthetic Llama-3-shaped decode linears (K x N) and sweeps.
WORKLOADS = {
    # single small matmul the fp64 oracle finishes in seconds
    0: {"M": [1], "shapes": [(4096, 4096)], "frac": [0.01], "dist": ["uniform"]},
    # Llama-3-8B decode linears: qkv, o, gate+up, down
    1: {"M": [1, 4, 8, 16],
        "shapes": [(4096, 6144), (4096, 4096), (4096, 28672), (14336, 4096)],
        "frac": [0.01], "dist": ["uniform"]},
    # density / structure sweep
    2: {"M": [8], "shapes": [(4096, 14336)],
        "frac": [0.0, 0.005, 0.01, 0.02, 0.05], "dist": ["uniform", "clustered"]},
    # Llama-3-70B decode linears
    3: {"M": [1, 8, 16, 32],
        "shapes": [(8192, 10240), (8192, 8192), (8192, 57344), (28672, 8192)],
        "frac": [0.01], "dist": ["uniform"]},
    # larger-batch crossover
    4: {"M": [32, 64, 128], "shapes": [(4096, 14336), (14336, 4096)],
        "frac": [0.01], "dist": ["uniform"]},
}

SHAPE_NAMES = {
    (4096, 6144): "qkv", (4096, 4096): "o", (4096, 28672): "gate_up",
    (14336, 4096): "down", (8192, 10240): "qkv70", (8192, 8192): "o70",
    (8192, 57344): "gate_up70", (28672, 8192): "down70",
    (4096, 14336): "k4096_n14336",
}


def seed_for(config: int, shape_idx: int, m_idx: int) -> int:
    """Seed rule: 1000*config + 10*shape_idx + M_idx."""
    return 1000 * config + 10 * shape_idx + m_idx


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return the bits.

    Used only to produce input bit patterns.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


@dataclass
class Problem:
    M: int
    K: int
    N: int
    group: int
    X: np.ndarray          # uint16 [M][K] bf16 bits
    Wq: np.ndarray         # uint32 [K/8][N]
    scales: np.ndarray     # uint16 [K/G][N] fp16 bits
    zeros: np.ndarray      # uint32 [K/G][N/8]
    k: np.ndarray          # int32 [nnz]
    n: np.ndarray          # int32 [nnz]
    v: np.ndarray          # uint16 [nnz] bf16 bits
    meta: dict = field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.k.shape[0])


def _pack_nibbles_along_axis0(codes: np.ndarray) -> np.ndarray:
    """codes uint8 [R][C] (R % 8 == 0) -> uint32 [R/8][C], row r in nibble r%8."""
    R, C = codes.shape
    c = codes.reshape(R // 8, 8, C)
    out = np.zeros((R // 8, C), dtype=np.uint32)
    for j in range(8):
        out |= c[:, j, :].astype(np.uint32) << np.uint32(4 * j)
    return out


def _pack_nibbles_along_axis1(codes: np.ndarray) -> np.ndarray:
    """codes uint8 [R][C] (C % 8 == 0) -> uint32 [R][C/8], column c in nibble c%8."""
    R, C = codes.shape
    c = codes.reshape(R, C // 8, 8)
    out = np.zeros((R, C // 8), dtype=np.uint32)
    for j in range(8):
        out |= c[:, :, j].astype(np.uint32) << np.uint32(4 * j)
    return out


def _draw_positions(rng, K, N, nnz, dist, cluster_frac, cluster_share):
    """Outlier positions as (k, n) int64 arrays, without replacement."""
    meta = {}
    if nnz == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64), meta
    if dist == "uniform":
        pos = rng.choice(K * N, size=nnz, replace=False)
        return pos // N, pos % N, meta
    if dist != "clustered":
        raise ValueError(f"unknown outlier distribution {dist!r}")
    n_c = int(round(cluster_frac * N))
    n_c = max(1, min(n_c, N - 1))
    cols = np.sort(rng.choice(N, size=n_c, replace=False))
    nnz_c = min(int(round(nnz * cluster_share)), n_c * K)
    rest = nnz - nnz_c
    if rest > (N - n_c) * K:
        raise ValueError("outlier request exceeds the matrix")
    p_c = rng.choice(n_c * K, size=nnz_c, replace=False)
    k_c, n_c_idx = p_c % K, cols[p_c // K]
    other = np.setdiff1d(np.arange(N), cols, assume_unique=True)
    p_o = rng.choice((N - n_c) * K, size=rest, replace=False)
    k_o, n_o = p_o % K, other[p_o // K]
    meta.update(clustered_columns=int(n_c), clustered_nnz=int(nnz_c),
                realised_share=float(nnz_c) / nnz)
    return np.concatenate([k_c, k_o]), np.concatenate([n_c_idx, n_o]), meta


def make_problem(M: int, K: int, N: int, frac: float = 0.01, seed: int = 0,
                 group: int = 128, dist: str = "uniform",
                 cluster_frac: float = 0.02, cluster_share: float = 0.5) -> Problem:
    """Random decode-linear problem.

    X ~ bf16(N(0,1)); codes uniform 0..15; scales fp16(U[0.005, 0.02));
    zero-points uniform 6..9; outliers: round(frac*K*N) positions without
    replacement, values bf16(0.5*N(0,1)) redrawn until |v| >= 0.1; the code at
    each outlier position is set to its group's zero-point.
    """
    if K % 8 or N % 8 or K % group:
        raise ValueError("K and N must be multiples of 8 and K of the group size")
    rng = np.random.Generator(np.random.PCG64(seed))
    X = bf16_bits_from_f32(rng.standard_normal((M, K), dtype=np.float32))
    codes = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    scales = rng.uniform(0.005, 0.02, size=(K // group, N)).astype(np.float16).view(np.uint16)
    z = rng.integers(6, 10, size=(K // group, N), dtype=np.uint8)
    nnz = int(round(frac * K * N))
    kk, nn, meta = _draw_positions(rng, K, N, nnz, dist, cluster_frac, cluster_share)
    v = _draw_values(rng, nnz)
    if nnz:
        codes[kk, nn] = z[kk // group, nn]
    meta.update(frac=frac, dist=dist, seed=seed)
    return Problem(M, K, N, group, X, _pack_nibbles_along_axis0(codes), scales,
                   _pack_nibbles_along_axis1(z), kk.astype(np.int32),
                   nn.astype(np.int32), v, meta)


def _draw_values(rng, nnz: int) -> np.ndarray:
    v = bf16_bits_from_f32((0.5 * rng.standard_normal(nnz)).astype(np.float32))
    while True:
        mag = (v.astype(np.uint32) << 16).view(np.float32)
        bad = np.flatnonzero(np.abs(mag) < 0.1)
        if bad.size == 0:
            return v
        v[bad] = bf16_bits_from_f32((0.5 * rng.standard_normal(bad.size)).astype(np.float32))


def make_exact_problem(M: int, K: int, N: int, frac: float = 0.01, seed: int = 0,
                       group: int = 128) -> Problem:
    """Problem whose every product and partial sum is exact in fp32.

    X integer in [-2, 2]; every scale 2^-4; outlier values +-j/8, j in 1..32;
    codes uniform 0..15 and zero-points uniform 6..9 as in make_problem.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    X = bf16_bits_from_f32(rng.integers(-2, 3, size=(M, K)).astype(np.float32))
    codes = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    scales = np.full((K // group, N), 0x2C00, dtype=np.uint16)   # fp16 0.0625
    z = rng.integers(6, 10, size=(K // group, N), dtype=np.uint8)
    nnz = int(round(frac * K * N))
    kk, nn, meta = _draw_positions(rng, K, N, nnz, "uniform", 0.0, 0.0)
    mags = rng.integers(1, 33, size=nnz).astype(np.float32) / 8.0
    signs = np.where(rng.integers(0, 2, size=nnz) == 1, -1.0, 1.0).astype(np.float32)
    v = bf16_bits_from_f32(mags * signs)
    if nnz:
        codes[kk, nn] = z[kk // group, nn]
    meta.update(frac=frac, dist="exact", seed=seed)
    return Problem(M, K, N, group, X, _pack_nibbles_along_axis0(codes), scales,
                   _pack_nibbles_along_axis1(z), kk.astype(np.int32),
                   nn.astype(np.int32), v, meta)


def make_activations(M: int, K: int, seed: int) -> np.ndarray:
    """bf16 bits of N(0,1) activations [M][K] (same recipe as make_problem's X)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return bf16_bits_from_f32(rng.standard_normal((M, K), dtype=np.float32))


def make_dense_weight(K: int, N: int, seed: int = 0, df: float = 4.0,
                      scale: float = 0.02) -> np.ndarray:
    """Synthetic dense fp32 weight [K][N] for the quantiser: scale * Student-t(df),
    heavy-tailed so that a small fraction of weights dominates the range."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return (scale * rng.standard_t(df, size=(K, N))).astype(np.float32)

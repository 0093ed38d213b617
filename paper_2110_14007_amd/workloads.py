"""Seeded synthetic workloads for the kNN / LOF outlier-detection path.

This module only draws random inputs; it holds none of the method's
arithmetic, so both the HIP path's callers and the oracle's tests may use it.

The paper evaluates on real tabular datasets and on synthetic data made of
Gaussian inliers plus uniform outliers (its appendix API example); those
datasets are not available here, so these five generators stand in for them.
Each draws in fp64 with numpy's PCG64 ``default_rng(seed)`` in the order
written below, casts to fp32 (round to nearest even) and shuffles rows with
the same generator.  Labels: 1 = outlier.

  C1  n=2,000    d=16  k=10  1,900 N(0, I) + 100 U[-6, 6]^16                 (kNN + LOF)
  C2  n=100,000  d=32  k=20  5 Gaussian components (means U[-10,10]^32,
                             isotropic std U[0.5, 2], 19,600 points each)
                             + 2,000 outliers uniform over the inlier bounding
                             box widened by 10 % of its width on each side    (kNN + LOF)
  C3  n=1,000,000 d=64 k=10  10 unit-variance Gaussian clusters (means 5*N(0,I),
                             99,000 points each) + 10,000 outliers 10*N(0, I) (kNN, fp16 filter,
                                                                               65,536-row query blocks)
  C4  n=200,000  d=512 k=50  rank-32 latent Z N(0, I_32) (199,000) x W, W = N(0,1)/sqrt(32)
                             (32 x 512), + 0.1*N(0, I) noise; 1,000 outliers N(0, I_512)
                                                                              (kNN, bf16 filter)
  C5  n=4,000,000 d=8  k=5   3,996,000 U[0,1]^8 + 4,000 U[1.5, 3]^8           (kNN)
  N1  n=30,000   d=200 phi=18  10 unit-variance Gaussian clusters (means 5*N(0,I),
                             2,970 points each) + 300 outliers 10*N(0, I);
                             phi = 0.9 sqrt(2d), 90 % of the typical distance
                             between two points of one cluster             (neighbours within range)
  L1  n=20,000   d=4   C2's recipe in 4 dimensions (5 Gaussian components, 19,600
                       points, 400 box outliers); sampling radii 0.5 * 5^(l/7),
                       l = 0..7 (0.5 to 2.5), alpha = 1/2, n_min = 20,
                       k_sigma = 3                                         (LOCI)

L1 is LOCI's workload: the detector is meant for low-dimensional data, where
counting neighbourhoods at half the sampling radius are not empty; its radii
span the clusters' scale (the median sampling neighbourhood grows from 17 to
3,300 points) and about 5.4e7 pairs lie within the largest.

N1 stands in for the paper's 30,000-sample synthetic set of its NWR runtime
breakdown (Table 5); the paper states neither its dimension nor its
threshold, so d follows the paper's other synthetic sets (200 features) and
phi is set relative to the cluster scale.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    d: int
    k: int
    seed: int
    # Filter precision the workload is specified with.  C1, C2 and C5 state
    # only the input type (fp32); the final lists are exact whatever the
    # filter, so those take the planner's choice ("auto").
    precision: str
    lof: bool  # whether the workload also asks for LOF
    query_block: int = 0  # 0 = planner's choice
    description: str = ""
    extra: dict = field(default_factory=dict)


WORKLOADS = {
    "C1": Workload("C1", 2_000, 16, 10, 1, "auto", True, 0,
                   "kNN-OD + LOF, n=2000 d=16 k=10: N(0,I) inliers + 5% U[-6,6] outliers"),
    "C2": Workload("C2", 100_000, 32, 20, 2, "auto", True, 0,
                   "kNN + LOF, n=100000 d=32 k=20: 5-Gaussian mixture + 2% uniform box outliers"),
    "C3": Workload("C3", 1_000_000, 64, 10, 3, "fp16", False, 65_536,
                   "kNN-OD, n=1000000 d=64 k=10: 10-cluster Gaussian mixture + 1% N(0,100I) "
                   "outliers, 65536-row query blocks, fp16 filter"),
    "C4": Workload("C4", 200_000, 512, 50, 4, "bf16", False, 0,
                   "kNN-OD, n=200000 d=512 k=50: rank-32 latent x projection + noise, 0.5% "
                   "full-rank outliers, bf16 filter"),
    "C5": Workload("C5", 4_000_000, 8, 5, 5, "auto", False, 0,
                   "kNN-OD, n=4000000 d=8 k=5: U[0,1]^8 + 0.1% U[1.5,3]^8 outliers"),
    "N1": Workload("N1", 30_000, 200, 0, 6, "fp16", False, 0,
                   "NWR, n=30000 d=200 phi=18: 10-cluster Gaussian mixture + 1% N(0,100I) "
                   "outliers, fp16 filter", {"phi": 18.0}),
    "L1": Workload("L1", 20_000, 4, 0, 7, "fp16", False, 0,
                   "LOCI, n=20000 d=4: 5-Gaussian mixture + 2% uniform box outliers, 8 radii "
                   "0.5..2.5, alpha 0.5, n_min 20, k_sigma 3",
                   {"radii": [0.5 * 5.0 ** (i / 7.0) for i in range(8)], "alpha": 0.5,
                    "n_min": 20, "k_sigma": 3.0}),
}


def _finish(rng, inliers: np.ndarray, outliers: np.ndarray):
    x = np.concatenate([inliers, outliers], axis=0)
    y = np.concatenate([np.zeros(len(inliers), np.int8), np.ones(len(outliers), np.int8)])
    x32 = x.astype(np.float32)
    perm = rng.permutation(len(x32))
    return np.ascontiguousarray(x32[perm]), y[perm]


def generate(name: str, n: int | None = None):
    """Return (X fp32 [n, d], labels int8 [n]) for workload ``name``.

    ``n`` optionally shrinks the workload (same recipe and proportions, fewer
    points) for quick tests.
    """
    w = WORKLOADS[name]
    n = w.n if n is None else int(n)
    rng = np.random.default_rng(w.seed)
    d = w.d
    if name == "C1":
        n_out = max(1, n * 100 // 2000)
        inl = rng.standard_normal((n - n_out, d))
        out = rng.uniform(-6.0, 6.0, (n_out, d))
    elif name in ("C2", "L1"):
        n_out = max(1, n * 2 // 100)
        n_in = n - n_out
        means = rng.uniform(-10.0, 10.0, (5, d))
        stds = rng.uniform(0.5, 2.0, 5)
        per = [n_in // 5 + (1 if c < n_in % 5 else 0) for c in range(5)]
        inl = np.concatenate([means[c] + stds[c] * rng.standard_normal((per[c], d))
                              for c in range(5)], axis=0)
        lo, hi = inl.min(axis=0), inl.max(axis=0)
        pad = 0.1 * (hi - lo)
        out = rng.uniform(lo - pad, hi + pad, (n_out, d))
    elif name in ("C3", "N1"):
        n_out = max(1, n // 100)
        n_in = n - n_out
        means = 5.0 * rng.standard_normal((10, d))
        per = [n_in // 10 + (1 if c < n_in % 10 else 0) for c in range(10)]
        inl = np.concatenate([means[c] + rng.standard_normal((per[c], d)) for c in range(10)],
                             axis=0)
        out = 10.0 * rng.standard_normal((n_out, d))
    elif name == "C4":
        n_out = max(1, n * 5 // 1000)
        n_in = n - n_out
        w_proj = rng.standard_normal((32, d)) / np.sqrt(32.0)
        z = rng.standard_normal((n_in, 32))
        inl = z @ w_proj + 0.1 * rng.standard_normal((n_in, d))
        out = rng.standard_normal((n_out, d))
    elif name == "C5":
        n_out = max(1, n // 1000)
        inl = rng.uniform(0.0, 1.0, (n - n_out, d))
        out = rng.uniform(1.5, 3.0, (n_out, d))
    else:
        raise KeyError(name)
    return _finish(rng, inl, out)


def sample_rows(name: str, n: int | None = None, count: int = 2048) -> np.ndarray:
    """Seeded query-row sample used to check large workloads row by row."""
    w = WORKLOADS[name]
    n = w.n if n is None else int(n)
    rng = np.random.default_rng((1000 if name[0] == "C" else 2000) + int(name[1:]))
    return np.sort(rng.choice(n, size=min(count, n), replace=False)).astype(np.int64)


def line(n: int = 10, d: int = 1) -> np.ndarray:
    """Points i * e_1, i = 0..n-1 (exact in every precision)."""
    x = np.zeros((n, d), np.float32)
    x[:, 0] = np.arange(n, dtype=np.float32)
    return x


def lattice(side: int = 9, dims: int = 2) -> np.ndarray:
    """Integer grid {0..side-1}^dims, row-major index (last coordinate fastest)."""
    axes = [np.arange(side, dtype=np.float32)] * dims
    grid = np.stack(np.meshgrid(*axes, indexing="ij"), axis=-1).reshape(-1, dims)
    return np.ascontiguousarray(grid)

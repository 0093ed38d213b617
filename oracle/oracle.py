"""Python front end of the fp64 CPU oracle (test infrastructure only).

Only ``tests/``, the smoke check and the CPU-baseline leg of the benchmark may
import this module.  It loads ``liboracle.so`` built from ``tod_oracle.c`` by
:func:`build` and exposes numpy-level wrappers.  Nothing here is shared with
the HIP path.

Functions:
  knn(xq, xr, k, exclude_self, rows=None) -> (idx int64 [m,k], dist fp64 [m,k])
  knn_self(x, k, rows=None)               -> kNN of X against itself, self excluded
  lof(idx, dist)                          -> (lof, lrd, kdist), fp64 [n]
  lof_rows(x, k, rows)                    -> (lof, lrd, kdist) for the listed rows
  lof_ties(x, k)                          -> (lof, lrd, kdist, count): LOF on Breunig's
                                             tie-inclusive k-distance neighbourhoods
  knn_score(dist, method="kth")           -> kNN outlier score from the k neighbour distances:
                                             k-th (default), mean, median or sum
  knn_vote(idx, labels, n_classes)        -> kNN classifier: majority label, ties to the smallest
  abod(x, idx)                            -> angle-based score: mean cosine over neighbour pairs
  cof(x, idx)                             -> (cof, acdist): connectivity-based outlier factor
  nwr(xq, xr, phi, exclude_self, rows=None) -> (row_ptr int64 [m+1], idx int64, dist fp64):
                                             neighbours within range, CSR, ascending index
  loci(x, radii, alpha, n_min, k_sigma)   -> LOCI (multi-granularity deviation factor) at a
                                             ladder of radii: counts, MDEF, sigma_MDEF,
                                             score and flag per point
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tod_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile tod_oracle.c with gcc (fp64, no fused multiply-add)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = [
            "gcc", "-O2", "-std=c11", "-D_GNU_SOURCE", "-ffp-contract=off", "-fno-fast-math",
            "-fPIC", "-shared", "-pthread", _SRC, "-o", tmp, "-lm",
        ]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    lib.oracle_knn.argtypes = [vp, i64, vp, i64, i64, i32, i32, vp, i64, i32, vp, vp]
    lib.oracle_knn.restype = ctypes.c_int
    lib.oracle_lof.argtypes = [i64, i32, vp, vp, vp, vp, vp]
    lib.oracle_lof.restype = ctypes.c_int
    lib.oracle_lof_rows.argtypes = [vp, i64, i64, i32, vp, i64, i32, vp, vp, vp]
    lib.oracle_lof_rows.restype = ctypes.c_int
    lib.oracle_nwr.argtypes = [vp, i64, vp, i64, i64, ctypes.c_double, i32, vp, i64, i32, vp, vp,
                               vp, vp]
    lib.oracle_nwr.restype = ctypes.c_int
    lib.oracle_default_threads.argtypes = []
    lib.oracle_default_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def default_threads() -> int:
    return int(_load().oracle_default_threads())


def _f32(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    if a.ndim != 2:
        raise ValueError("expected a 2-D array")
    return a


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def knn(xq, xr, k: int, exclude_self: bool = False, rows=None, threads: int = 0):
    """k nearest references of each query row, sorted by (distance, index)."""
    xq, xr = _f32(xq), _f32(xr)
    if xq.shape[1] != xr.shape[1]:
        raise ValueError("dimension mismatch")
    lib = _load()
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        m = rows.shape[0]
    else:
        m = xq.shape[0]
    idx = np.empty((m, k), dtype=np.int64)
    dist = np.empty((m, k), dtype=np.float64)
    rc = lib.oracle_knn(
        _ptr(xq), xq.shape[0], _ptr(xr), xr.shape[0], xq.shape[1], int(k), int(bool(exclude_self)),
        _ptr(rows) if rows is not None else None, m, int(threads), _ptr(idx), _ptr(dist))
    if rc != 0:
        raise ValueError("oracle_knn rejected its arguments (rc=%d)" % rc)
    return idx, dist


def knn_self(x, k: int, rows=None, threads: int = 0):
    """kNN of X against itself with each point's own row excluded."""
    return knn(x, x, k, exclude_self=True, rows=rows, threads=threads)


def knn_score(dist, method: str = "kth") -> np.ndarray:
    """kNN outlier score of each row from its k neighbour distances (sorted
    ascending, fp64): the distance to the k-th nearest neighbour (Table 1's
    kNN detector), or the mean, the median (mean of the two middle distances
    for even k) or the sum of the k distances (the weight of Angiulli and
    Pizzuti's detector, which the paper cites for kNN)."""
    d = np.asarray(dist, dtype=np.float64)
    if method in ("kth", "largest"):
        return d[:, -1].copy()
    if method == "mean":
        return d.sum(axis=1) / d.shape[1]
    if method == "median":
        return np.median(d, axis=1)
    if method == "sum":
        return d.sum(axis=1)
    raise ValueError("unknown score method %r" % method)


def abod(x, idx) -> np.ndarray:
    """Angle-based outlier score (Section 4.3's ABOD built from the kNN and
    cosine-similarity operators): for point i with neighbours N_k(i), the
    mean over the unordered pairs {b, c} of distinct neighbours of the cosine
    of the angle between x_b - x_i and x_c - x_i.  Differences, dot products
    and norms in fp64, dot products summed over the columns in order; pairs
    with a zero-length difference (a duplicate of x_i) are left out, and a
    point without any pair left scores 0.  Higher means more outlying (the
    neighbours lie in one direction)."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    idx = np.asarray(idx, dtype=np.int64)
    n, k = idx.shape
    out = np.zeros(n, dtype=np.float64)
    for i in range(n):
        v = x[idx[i]] - x[i]                       # k x d, exact differences
        g = np.zeros((k, k), dtype=np.float64)
        for t in range(v.shape[1]):                # column order, as the definition sums
            g += np.outer(v[:, t], v[:, t])
        total, count = 0.0, 0
        for b in range(k):
            for c in range(b + 1, k):
                if g[b, b] > 0.0 and g[c, c] > 0.0:
                    total += g[b, c] / np.sqrt(g[b, b] * g[c, c])
                    count += 1
        out[i] = total / count if count else 0.0
    return out


def cof(x, idx):
    """Connectivity-based outlier factor (Tang et al., one of Table 1's
    proximity-based detectors), from the kNN lists.

    For point p with neighbours N_k(p): the set-based nearest path over
    G = {p} + N_k(p) starts from S = {p} and adds, k times, the point of G
    outside S nearest to S (distance to a set = smallest distance to a
    member; ties to the lower row index); the i-th step costs that
    distance c_i.  The average chaining distance is
        ac(p) = sum_i 2 (k + 1 - i) / (k (k + 1)) * c_i,
    and COF(p) = (ac(p) + 1e-10) / (mean over o in N_k(p) of ac(o) + 1e-10)
    (the 1e-10 keeps duplicates finite, as LOF's lrd does).  Squared
    distances are the fp64 sums of the definition, compared squared, and
    their square roots are the costs.  Returns (cof, ac), fp64."""
    xd = np.asarray(x, dtype=np.float32).astype(np.float64)
    idx = np.asarray(idx, dtype=np.int64)
    n, k = idx.shape
    ac = np.zeros(n, dtype=np.float64)
    for p in range(n):
        g = [p] + idx[p].tolist()
        rows = xd[g]
        d2 = np.zeros((k + 1, k + 1), dtype=np.float64)
        for t in range(rows.shape[1]):  # every pair summed over the columns in order
            e = rows[:, t][:, None] - rows[:, t][None, :]
            d2 = d2 + e * e
        in_s = [True] + [False] * k
        best = [d2[0][j] for j in range(k + 1)]
        total = 0.0
        for i in range(1, k + 1):
            cand = [j for j in range(k + 1) if not in_s[j]]
            o = min(cand, key=lambda j: (best[j], g[j]))
            total = total + 2.0 * (k + 1 - i) / (k * (k + 1)) * np.sqrt(best[o])
            in_s[o] = True
            for j in range(k + 1):
                if not in_s[j] and d2[o][j] < best[j]:
                    best[j] = d2[o][j]
        ac[p] = total
    mean_nb = np.array([sum(ac[o] for o in idx[p].tolist()) / k for p in range(n)])
    return (ac + 1e-10) / (mean_nb + 1e-10), ac


def sq_dist_matrix(x) -> np.ndarray:
    """All pairwise squared distances of the rows of X in fp64, each the sum
    over the columns in order of ((double)x_pt - (double)x_qt)^2 (the
    definition, no fused multiply-add)."""
    xd = np.asarray(x, dtype=np.float32).astype(np.float64)
    n, d = xd.shape
    d2 = np.zeros((n, n), dtype=np.float64)
    for t in range(d):
        e = xd[:, t][:, None] - xd[:, t][None, :]
        d2 = d2 + e * e
    return d2


def loci(x, radii, alpha: float = 0.5, n_min: int = 20, k_sigma: float = 3.0):
    """LOCI (Papadimitriou et al., ICDE 2003; Table 1's proximity-based
    detector built, like LOF, on neighbours within range) at a ladder of
    sampling radii r_1 < ... < r_L.

    With N(p, r) = {q : d(p, q) <= r} (p itself included) and n(p, r) its size:
      counting neighbourhood size   n(p, alpha r)
      sampling neighbourhood size   n(p, r)
      n_hat(p, r)   = mean over q in N(p, r) of n(q, alpha r)
      sigma_n(p, r) = standard deviation (population) of the same values
      MDEF(p, r)       = 1 - n(p, alpha r) / n_hat(p, r)
      sigma_MDEF(p, r) = sigma_n(p, r) / n_hat(p, r).
    A radius counts for p when n(p, r) >= n_min; p is flagged when
    MDEF > k_sigma * sigma_MDEF at some counted radius, and its score is the
    largest MDEF / sigma_MDEF over the counted radii (0 where sigma_MDEF is 0,
    which forces MDEF = 0 since p samples itself; 0 when no radius counts).

    Membership is exact: d(p, q) <= r iff the fp64 squared distance of the
    definition is <= fl(r * r), and d(p, q) <= alpha r iff it is <=
    fl(fl(alpha * r)^2).  The neighbourhood sums are exact integers; then, in
    fp64 and in this order: n_hat = S1 / n_r, var = S2 / n_r - n_hat * n_hat
    (negative values to 0), sigma_n = sqrt(var), MDEF = 1 - n_a / n_hat,
    sigma_MDEF = sigma_n / n_hat.

    Returns a dict of n_alpha, n_r (int64 [n, L]), mdef, sigma_mdef (fp64
    [n, L]), score (fp64 [n]) and flag (bool [n])."""
    radii = np.asarray(radii, dtype=np.float64)
    if radii.ndim != 1 or radii.size < 1 or np.any(np.diff(radii) <= 0) or radii[0] < 0:
        raise ValueError("radii must be a non-empty strictly increasing list of values >= 0")
    d2 = sq_dist_matrix(x)
    n = d2.shape[0]
    nl = radii.size
    r2 = radii * radii
    a2 = (np.float64(alpha) * radii) ** 2
    n_a = np.zeros((n, nl), dtype=np.int64)
    n_r = np.zeros((n, nl), dtype=np.int64)
    s1 = np.zeros((n, nl), dtype=np.int64)
    s2 = np.zeros((n, nl), dtype=np.int64)
    for l in range(nl):
        n_a[:, l] = (d2 <= a2[l]).sum(axis=1)
    for l in range(nl):
        samp = (d2 <= r2[l]).astype(np.int64)
        n_r[:, l] = samp.sum(axis=1)
        s1[:, l] = samp @ n_a[:, l]
        s2[:, l] = samp @ (n_a[:, l] * n_a[:, l])
    nr_f = n_r.astype(np.float64)
    n_hat = s1.astype(np.float64) / nr_f
    var = s2.astype(np.float64) / nr_f - n_hat * n_hat
    var = np.where(var < 0.0, 0.0, var)
    sigma_n = np.sqrt(var)
    mdef = 1.0 - n_a.astype(np.float64) / n_hat
    sigma_mdef = sigma_n / n_hat
    counted = n_r >= int(n_min)
    ratio = np.where(sigma_mdef > 0.0, mdef / np.where(sigma_mdef > 0.0, sigma_mdef, 1.0), 0.0)
    score = np.where(counted, ratio, -np.inf).max(axis=1)
    score = np.where(counted.any(axis=1), score, 0.0)
    flag = (counted & (mdef > np.float64(k_sigma) * sigma_mdef)).any(axis=1)
    return {"n_alpha": n_a, "n_r": n_r, "mdef": mdef, "sigma_mdef": sigma_mdef,
            "score": score, "flag": flag}


def knn_vote(idx, labels, n_classes: int) -> np.ndarray:
    """kNN classifier (Appendix B): for each row, the most frequent label among
    its k neighbours; ties go to the smallest label."""
    idx = np.asarray(idx, dtype=np.int64)
    lab = np.asarray(labels, dtype=np.int64)[idx]  # [m, k]
    counts = np.zeros((lab.shape[0], int(n_classes)), dtype=np.int64)
    np.add.at(counts, (np.repeat(np.arange(lab.shape[0]), lab.shape[1]), lab.ravel()), 1)
    return counts.argmax(axis=1).astype(np.int32)  # argmax returns the first (smallest) maximum


def lof(idx, dist):
    """LOF of every point from complete kNN lists; returns (lof, lrd, kdist)."""
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    dist = np.ascontiguousarray(dist, dtype=np.float64)
    n, k = idx.shape
    out = [np.empty(n, dtype=np.float64) for _ in range(3)]
    rc = _load().oracle_lof(n, k, _ptr(idx), _ptr(dist), _ptr(out[2]), _ptr(out[1]), _ptr(out[0]))
    if rc != 0:
        raise ValueError("oracle_lof failed (rc=%d)" % rc)
    return out[0], out[1], out[2]


def lof_ties(x, k: int):
    """LOF on Breunig et al.'s k-distance neighbourhoods, which keep every point
    tied at the k-distance (so a neighbourhood can hold more than k points);
    each point's own row excluded.  LOF is one of Table 1's detectors and, like
    LOCI, a user of neighbours within range (Section 5.3): N_k(p) is the range
    query around p at radius kdist(p).

      D2(p, o)   fp64 sum over the columns in order of ((double)x_pt - (double)x_ot)^2
      kd2(p)     the k-th smallest D2(p, o) over o != p
      N_k(p)   = {o != p : D2(p, o) <= kd2(p)}
      kdist(p) = sqrt(kd2(p)),  D(p, o) = sqrt(D2(p, o))
      reach(p, o) = max(kdist(o), D(p, o))
      lrd(p)   = 1 / (sum_{o in N_k(p)} reach(p, o) / |N_k(p)| + 1e-10)
      LOF(p)   = (sum_{o in N_k(p)} lrd(o) / |N_k(p)|) / lrd(p)

    Plain n x n evaluation (memory n^2 fp64): for small point sets.
    Returns (lof, lrd, kdist, count) with count[p] = |N_k(p)|."""
    d2 = sq_dist_matrix(x)
    n = d2.shape[0]
    k = int(k)
    if not 1 <= k < n:
        raise ValueError("lof_ties needs 1 <= k < n")
    np.fill_diagonal(d2, np.inf)  # o != p
    kd2 = np.sort(d2, axis=1)[:, k - 1]
    kdist = np.sqrt(kd2)
    members = [np.nonzero(d2[p] <= kd2[p])[0] for p in range(n)]
    count = np.array([m.size for m in members], dtype=np.int64)
    lrd = np.empty(n, dtype=np.float64)
    for p in range(n):
        m = members[p]
        reach = np.maximum(kdist[m], np.sqrt(d2[p, m]))
        lrd[p] = 1.0 / (reach.sum() / m.size + 1e-10)
    lof_v = np.empty(n, dtype=np.float64)
    for p in range(n):
        m = members[p]
        lof_v[p] = (lrd[m].sum() / m.size) / lrd[p]
    return lof_v, lrd, kdist, count


def lof_rows(x, k: int, rows, threads: int = 0):
    """LOF of the listed rows of X, computed from their 2-hop neighbourhoods."""
    x = _f32(x)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    m = rows.shape[0]
    out = [np.empty(m, dtype=np.float64) for _ in range(3)]
    rc = _load().oracle_lof_rows(_ptr(x), x.shape[0], x.shape[1], int(k), _ptr(rows), m,
                                 int(threads), _ptr(out[0]), _ptr(out[1]), _ptr(out[2]))
    if rc != 0:
        raise ValueError("oracle_lof_rows failed (rc=%d)" % rc)
    return out[0], out[1], out[2]


def nwr(xq, xr, phi: float, exclude_self: bool = False, rows=None, threads: int = 0):
    """Neighbours within range phi (a radius) of each query row, as CSR.

    A pair is in range iff its fp64 squared distance is <= phi * phi; each
    row lists its references in increasing index.
    """
    xq, xr = _f32(xq), _f32(xr)
    if xq.shape[1] != xr.shape[1]:
        raise ValueError("dimension mismatch")
    lib = _load()
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        m = rows.shape[0]
    else:
        m = xq.shape[0]
    rp = _ptr(rows) if rows is not None else None
    counts = np.empty(m, dtype=np.int64)
    rc = lib.oracle_nwr(_ptr(xq), xq.shape[0], _ptr(xr), xr.shape[0], xq.shape[1], float(phi),
                        int(bool(exclude_self)), rp, m, int(threads), _ptr(counts), None, None, None)
    if rc != 0:
        raise ValueError("oracle_nwr rejected its arguments (rc=%d)" % rc)
    row_ptr = np.zeros(m + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    nnz = int(row_ptr[-1])
    idx = np.empty(max(nnz, 1), dtype=np.int64)
    dist = np.empty(max(nnz, 1), dtype=np.float64)
    rc = lib.oracle_nwr(_ptr(xq), xq.shape[0], _ptr(xr), xr.shape[0], xq.shape[1], float(phi),
                        int(bool(exclude_self)), rp, m, int(threads), None, _ptr(row_ptr),
                        _ptr(idx), _ptr(dist))
    if rc != 0:
        raise ValueError("oracle_nwr fill failed (rc=%d)" % rc)
    return row_ptr, idx[:nnz], dist[:nnz]

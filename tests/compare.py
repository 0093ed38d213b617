"""Comparison of HIP-path results with the oracle's.

Neighbour indices must match position by position.  A mismatch at rank p is
excused (and counted) only when the two candidates are an oracle near-tie:
the fp64 distance from the query to the HIP path's neighbour is within 1e-6
relative of the oracle's p-th distance.  Pins built from integer data pass
``allow_ties=False``, which excuses nothing.  Distances and scores must
agree within 1e-5 relative (exactly 0 where the oracle's is 0).
"""
from __future__ import annotations

import numpy as np

REL_TIE = 1e-6
REL_VAL = 1e-5


def compare_knn(xq, xr, rows, idx_gpu, dist_gpu, idx_or, dist_or, allow_ties=True):
    """Returns (n_excused, excused_rows).  Raises AssertionError on a real mismatch."""
    idx_gpu = np.asarray(idx_gpu)
    dist_gpu = np.asarray(dist_gpu, dtype=np.float64)
    rows = np.asarray(rows)
    assert idx_gpu.shape == idx_or.shape, (idx_gpu.shape, idx_or.shape)
    bad = idx_gpu != idx_or
    excused_rows = set()
    n_excused = 0
    if bad.any():
        r, p = np.nonzero(bad)
        if not allow_ties:
            raise AssertionError("index mismatch at %d positions (first: row %d rank %d: "
                                 "%d vs %d)" % (len(r), rows[r[0]], p[0], idx_gpu[r[0], p[0]],
                                                idx_or[r[0], p[0]]))
        assert np.all((idx_gpu[r, p] >= 0) & (idx_gpu[r, p] < xr.shape[0]))
        d_alt = np.sqrt(((xq[rows[r]].astype(np.float64) -
                          xr[idx_gpu[r, p]].astype(np.float64)) ** 2).sum(axis=1))
        ref = dist_or[r, p]
        ok = np.abs(d_alt - ref) <= REL_TIE * np.maximum(ref, 1e-300)
        if not ok.all():
            i = np.nonzero(~ok)[0][0]
            raise AssertionError(
                "index mismatch at row %d rank %d: gpu %d (D=%.17g) vs oracle %d (D=%.17g)" %
                (rows[r[i]], p[i], idx_gpu[r[i], p[i]], d_alt[i], idx_or[r[i], p[i]], ref[i]))
        n_excused = int(ok.sum())
        excused_rows = set(rows[r].tolist())
    zero = dist_or == 0
    assert np.all(dist_gpu[zero] == 0), "distance must be exactly 0 where the oracle's is"
    rel = np.abs(dist_gpu - dist_or) / np.where(zero, 1.0, dist_or)
    assert np.all(rel <= REL_VAL), "distance rel err %.3g" % rel.max()
    return n_excused, excused_rows


def compare_scores(got, want, rows=None, excused_rows=(), what="score"):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    keep = np.ones(len(want), bool)
    if rows is not None and excused_rows:
        keep = ~np.isin(np.asarray(rows), list(excused_rows))
    g, w = got[keep], want[keep]
    zero = w == 0
    assert np.all(g[zero] == 0), what
    rel = np.abs(g - w) / np.where(zero, 1.0, np.abs(w))
    assert np.all(rel <= REL_VAL), "%s rel err %.3g at %d" % (what, rel.max(), int(np.argmax(rel)))
    return int((~keep).sum())

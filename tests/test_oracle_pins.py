"""Pins for the fp64 CPU oracle: it is checked against hand-derived values,
exact rational brute force, closed forms and invariances, never against
itself or the HIP path."""
import math
import os
import statistics
from fractions import Fraction

import numpy as np
import pytest

from paper_2110_14007_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _parse_line_fixture():
    out = {}
    with open(os.path.join(GOLDEN, "line10.txt")) as f:
        for raw in f:
            raw = raw.strip()
            if not raw or raw.startswith("#"):
                continue
            parts = raw.split()
            k, field, vals = int(parts[0]), parts[1], parts[2:]
            assert len(vals) == 10
            if field == "idx":
                out[(k, field)] = [[int(t) for t in v.split(",")] for v in vals]
            else:
                out[(k, field)] = [Fraction(v) for v in vals]
    return out


@pytest.mark.parametrize("k", [2, 3])
@pytest.mark.parametrize("d", [1, 4])
def test_line_golden(oracle_mod, k, d):
    gold = _parse_line_fixture()
    x = workloads.line(10, d)
    idx, dist = oracle_mod.knn_self(x, k)
    assert idx.tolist() == gold[(k, "idx")]
    assert dist[:, -1].tolist() == [float(v) for v in gold[(k, "kdist")]]
    lof, lrd, kdist = oracle_mod.lof(idx, dist)
    np.testing.assert_array_equal(kdist, [float(v) for v in gold[(k, "kdist")]])
    np.testing.assert_allclose(lrd, [float(v) for v in gold[(k, "lrd")]], rtol=1e-9)
    np.testing.assert_allclose(lof, [float(v) for v in gold[(k, "lof")]], rtol=1e-9)
    # The kNN-OD score is the distance to the k-th neighbour.
    np.testing.assert_array_equal(oracle_mod.knn_score(dist), kdist)


def _steps_from_boundary(side, coords):
    return np.minimum(coords, side - 1 - coords).min(axis=1)


@pytest.mark.parametrize("k", [4, 8])
def test_lattice_closed_forms(oracle_mod, k):
    side = 9
    x = workloads.lattice(side, 2)
    idx, dist = oracle_mod.knn_self(x, k)
    lof, lrd, kdist = oracle_mod.lof(idx, dist)
    depth = _steps_from_boundary(side, x.astype(int))
    r, c = x[:, 0].astype(int), x[:, 1].astype(int)
    on_row_edge = (r == 0) | (r == side - 1)
    on_col_edge = (c == 0) | (c == side - 1)
    corner = on_row_edge & on_col_edge
    edge = (on_row_edge | on_col_edge) & ~corner
    interior = depth >= 1
    if k == 4:
        # 4 axis neighbours at 1; an edge point has 3 at 1 then diagonals at
        # sqrt(2); a corner has 2 at 1, one at sqrt(2), then two at 2.
        np.testing.assert_array_equal(kdist[interior], 1.0)
        np.testing.assert_array_equal(kdist[edge], math.sqrt(2.0))
        np.testing.assert_array_equal(kdist[corner], 2.0)
    else:
        # 4 at distance 1 and 4 diagonals at sqrt(2) fill k = 8 exactly.
        np.testing.assert_array_equal(kdist[interior], math.sqrt(2.0))
    # LOF = 1 wherever the two-hop neighbourhood sees no boundary effect.
    deep = depth >= 3
    assert deep.sum() == 9
    np.testing.assert_allclose(lof[deep], 1.0, rtol=0, atol=1e-12)
    assert np.all(np.abs(lof[~deep] - 1.0) > 1e-6)


def test_lattice_tiebreak_k5(oracle_mod):
    x = workloads.lattice(9, 2)
    idx, dist = oracle_mod.knn_self(x, 5)
    p = 4 * 9 + 4
    # Axis neighbours (3,4),(4,3),(4,5),(5,4) at 1, then the lowest-index
    # diagonal (3,3) among four tied at sqrt(2).
    assert idx[p].tolist() == [31, 39, 41, 49, 30]
    np.testing.assert_array_equal(dist[p], [1, 1, 1, 1, math.sqrt(2.0)])


def test_lattice_3d_k6(oracle_mod):
    side = 7
    x = workloads.lattice(side, 3)
    idx, dist = oracle_mod.knn_self(x, 6)
    lof, _, kdist = oracle_mod.lof(idx, dist)
    depth = _steps_from_boundary(side, x.astype(int))
    np.testing.assert_array_equal(kdist[depth >= 1], 1.0)
    np.testing.assert_allclose(lof[depth >= 3], 1.0, rtol=0, atol=1e-12)
    assert np.all(np.abs(lof[depth < 3] - 1.0) > 1e-6)


def _exact_knn(xq, xr, k, exclude_self):
    """Exact rational brute force: every fp32 value is a dyadic rational."""
    fq = [[Fraction(float(v)) for v in row] for row in xq]
    fr = [[Fraction(float(v)) for v in row] for row in xr]
    idx, dist = [], []
    for i, q in enumerate(fq):
        cand = []
        for j, r in enumerate(fr):
            if exclude_self and i == j:
                continue
            cand.append((sum((a - b) * (a - b) for a, b in zip(q, r)), j))
        cand.sort()
        idx.append([j for _, j in cand[:k]])
        dist.append([math.sqrt(float(d2)) for d2, _ in cand[:k]])
    return np.array(idx), np.array(dist)


def _tiny_cases():
    rng = np.random.default_rng(12345)
    cases = []
    for case in range(24):
        n = int(rng.integers(2, 51))
        d = int(rng.choice([1, 2, 3, 8]))
        kind = case % 3
        if kind == 0:
            x = rng.standard_normal((n, d)).astype(np.float32)
        elif kind == 1:  # small integers: many exact ties
            x = rng.integers(-3, 4, (n, d)).astype(np.float32)
        else:  # wide dynamic range, duplicates
            x = (rng.standard_normal((n, d)) * 10.0 ** rng.integers(-3, 4, (n, 1))).astype(
                np.float32)
            x[n // 2] = x[0]
        k = int(rng.integers(1, n))  # 1 .. n-1
        cases.append((x, k))
    return cases


@pytest.mark.parametrize("case", range(24))
def test_exact_rational_bruteforce_self(oracle_mod, case):
    x, k = _tiny_cases()[case]
    ei, ed = _exact_knn(x, x, k, True)
    idx, dist = oracle_mod.knn_self(x, k)
    np.testing.assert_array_equal(idx, ei)
    np.testing.assert_allclose(dist, ed, rtol=1e-14, atol=0)


@pytest.mark.parametrize("case", range(8))
def test_exact_rational_bruteforce_cross(oracle_mod, case):
    rng = np.random.default_rng(777 + case)
    nq, nr = int(rng.integers(1, 30)), int(rng.integers(1, 40))
    d = int(rng.choice([1, 3, 8]))
    xq = rng.integers(-2, 3, (nq, d)).astype(np.float32) if case % 2 else \
        rng.standard_normal((nq, d)).astype(np.float32)
    xr = rng.integers(-2, 3, (nr, d)).astype(np.float32) if case % 2 else \
        rng.standard_normal((nr, d)).astype(np.float32)
    k = int(rng.integers(1, nr + 1))
    ei, ed = _exact_knn(xq, xr, k, False)
    idx, dist = oracle_mod.knn(xq, xr, k)
    np.testing.assert_array_equal(idx, ei)
    np.testing.assert_allclose(dist, ed, rtol=1e-14, atol=0)


def test_one_dimensional_sorted_neighbours(oracle_mod):
    # In 1-D the k nearest neighbours of a point are a contiguous window of
    # the sorted order; check the oracle against that textbook property.
    rng = np.random.default_rng(5)
    v = rng.permutation(np.arange(200, dtype=np.float32) * 0.37 + rng.random(200).astype(
        np.float32) * 0.01)
    x = v[:, None].astype(np.float32)
    k = 7
    idx, _ = oracle_mod.knn_self(x, k)
    order = np.argsort(v, kind="stable")
    rank = np.empty_like(order)
    rank[order] = np.arange(len(v))
    for i in range(len(v)):
        ranks = np.sort(rank[idx[i]])
        window = np.concatenate([ranks, [rank[i]]])
        window.sort()
        assert window[-1] - window[0] == k  # k neighbours + self are contiguous


def test_permutation_invariance(oracle_mod):
    rng = np.random.default_rng(99)
    x = rng.standard_normal((300, 5)).astype(np.float32)
    perm = rng.permutation(300)
    k = 6
    idx, dist = oracle_mod.knn_self(x, k)
    lof, _, _ = oracle_mod.lof(idx, dist)
    pidx, pdist = oracle_mod.knn_self(x[perm], k)
    plof, _, _ = oracle_mod.lof(pidx, pdist)
    # row r of the permuted problem is original row perm[r]
    np.testing.assert_array_equal(perm[pidx], idx[perm])
    np.testing.assert_array_equal(pdist, dist[perm])
    np.testing.assert_allclose(plof, lof[perm], rtol=1e-13)


def test_power_of_two_scaling(oracle_mod):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((250, 7)).astype(np.float32)
    k = 5
    idx, dist = oracle_mod.knn_self(x, k)
    lof, _, _ = oracle_mod.lof(idx, dist)
    sidx, sdist = oracle_mod.knn_self(x * np.float32(64.0), k)
    slof, _, _ = oracle_mod.lof(sidx, sdist)
    np.testing.assert_array_equal(sidx, idx)
    np.testing.assert_array_equal(sdist, dist * 64.0)
    np.testing.assert_allclose(slof, lof, rtol=1e-8)


def test_duplicates_convention(oracle_mod):
    # Two coincident points are each other's 1-NN at distance 0: reach is 0
    # and the 1e-10 guard gives lrd = 1e10 instead of a division by zero.
    x = np.array([[0, 0], [0, 0], [5, 0], [5, 1], [9, 9]], np.float32)
    idx, dist = oracle_mod.knn_self(x, 1)
    assert idx[:2, 0].tolist() == [1, 0]
    lof, lrd, kdist = oracle_mod.lof(idx, dist)
    assert kdist[0] == 0.0 and kdist[1] == 0.0
    np.testing.assert_allclose(lrd[:2], 1e10)
    np.testing.assert_allclose(lof[:2], 1.0)
    assert np.all(np.isfinite(lof))


def test_lof_rows_matches_full_lists(oracle_mod):
    x, _ = workloads.generate("C1")
    k = 10
    idx, dist = oracle_mod.knn_self(x, k)
    lof, lrd, kdist = oracle_mod.lof(idx, dist)
    rows = workloads.sample_rows("C1", count=64)
    rl, rlrd, rk = oracle_mod.lof_rows(x, k, rows)
    np.testing.assert_array_equal(rk, kdist[rows])
    np.testing.assert_array_equal(rlrd, lrd[rows])
    np.testing.assert_array_equal(rl, lof[rows])


def test_outliers_score_high(oracle_mod):
    # Sanity only (no published value): on C1 the uniform outliers should
    # dominate the top of both rankings.
    x, y = workloads.generate("C1")
    idx, dist = oracle_mod.knn_self(x, 10)
    score = oracle_mod.knn_score(dist)
    lof, _, _ = oracle_mod.lof(idx, dist)
    top = np.argsort(-score)[:100]
    assert y[top].mean() > 0.9
    top = np.argsort(-lof)[:100]
    assert y[top].mean() > 0.8


def test_oracle_rejects_bad_arguments(oracle_mod):
    x = np.zeros((5, 2), np.float32)
    with pytest.raises(ValueError):
        oracle_mod.knn_self(x, 5)  # k > n - 1
    with pytest.raises(ValueError):
        oracle_mod.knn(x, x, 0)


def test_workload_shapes_small():
    for name in ("C1", "C2", "C3", "C4", "C5"):
        x, y = workloads.generate(name, n=3000)
        w = workloads.WORKLOADS[name]
        assert x.shape == (3000, w.d) and x.dtype == np.float32
        assert y.shape == (3000,) and 0 < y.sum() < 3000
        x2, _ = workloads.generate(name, n=3000)
        np.testing.assert_array_equal(x, x2)


# ---------------------------------------------------------------------------
# Neighbours within range (NWR, Section 5.3): phi is a radius, a pair is in
# range iff its squared distance is <= phi^2.
# ---------------------------------------------------------------------------

def _nwr_lists(row_ptr, idx):
    return [idx[row_ptr[i]:row_ptr[i + 1]].tolist() for i in range(len(row_ptr) - 1)]


@pytest.mark.parametrize("phi,offsets", [
    (1.0, [(0, 0), (1, 0), (-1, 0), (0, 1), (0, -1)]),           # boundary pairs (D = 1) count
    (1.25, [(0, 0), (1, 0), (-1, 0), (0, 1), (0, -1)]),          # between 1 and sqrt 2
    (math.sqrt(2.0), [(a, b) for a in (-1, 0, 1) for b in (-1, 0, 1)]),  # fl(sqrt2)^2 > 2
    (1.5, [(a, b) for a in (-1, 0, 1) for b in (-1, 0, 1)]),
    (2.0, [(a, b) for a in (-2, -1, 0, 1, 2) for b in (-2, -1, 0, 1, 2) if a * a + b * b <= 4]),
    (0.999, [(0, 0)]),
])
@pytest.mark.parametrize("excl", [False, True])
def test_nwr_lattice_closed_forms(oracle_mod, phi, offsets, excl):
    side = 9
    x = workloads.lattice(side, 2)
    rp, idx, dist = oracle_mod.nwr(x, x, phi, exclude_self=excl)
    coords = x.astype(int)
    pos = {tuple(c): i for i, c in enumerate(coords.tolist())}
    for i, (r, c) in enumerate(coords.tolist()):
        want = sorted(pos[(r + a, c + b)] for a, b in offsets
                      if (r + a, c + b) in pos and not (excl and a == 0 and b == 0))
        got = idx[rp[i]:rp[i + 1]].tolist()
        assert got == want, (i, got, want)
        np.testing.assert_array_equal(
            dist[rp[i]:rp[i + 1]],
            [math.sqrt((coords[j][0] - r) ** 2 + (coords[j][1] - c) ** 2) for j in want])


@pytest.mark.parametrize("d", [1, 4])
def test_nwr_line_windows(oracle_mod, d):
    x = workloads.line(10, d)
    rp, idx, _ = oracle_mod.nwr(x, x, 2.0, exclude_self=True)
    assert _nwr_lists(rp, idx) == [[j for j in range(max(0, i - 2), min(10, i + 3)) if j != i]
                                   for i in range(10)]


def _exact_nwr(xq, xr, phi2, exclude_self):
    fq = [[Fraction(float(v)) for v in row] for row in xq]
    fr = [[Fraction(float(v)) for v in row] for row in xr]
    out = []
    for i, q in enumerate(fq):
        out.append([j for j, r in enumerate(fr) if not (exclude_self and i == j)
                    and sum((a - b) * (a - b) for a, b in zip(q, r)) <= phi2])
    return out


@pytest.mark.parametrize("case", range(24))
def test_nwr_exact_rational_bruteforce(oracle_mod, case):
    x, _ = _tiny_cases()[case]
    fx = [[Fraction(float(v)) for v in row] for row in x]
    d2 = sorted({sum((a - b) * (a - b) for a, b in zip(p, q)) for p in fx for q in fx})
    # A radius strictly inside a gap between two exact squared distances, far
    # from both relative to fp64 rounding, so that the fp64 decision is exact.
    gaps = [(b - a, a, b) for a, b in zip(d2, d2[1:]) if b - a > Fraction(1, 10 ** 6) * b]
    _, lo, hi = gaps[len(gaps) // 2]
    mid = (lo + hi) / 2
    phi = math.sqrt(float(mid))
    for excl in (False, True):
        rp, idx, _ = oracle_mod.nwr(x, x, phi, exclude_self=excl)
        assert _nwr_lists(rp, idx) == _exact_nwr(x, x, mid, excl)


def test_nwr_contains_knn(oracle_mod):
    x, _ = workloads.generate("C1")
    k = 10
    kidx, kdist = oracle_mod.knn_self(x, k)
    r = kdist[:, -1]
    rows = np.arange(0, len(x), 7)
    for i in rows:
        rp, idx, _ = oracle_mod.nwr(x, x, float(r[i]) * (1 + 1e-9), exclude_self=True, rows=[i])
        got = set(idx.tolist())
        assert set(kidx[i].tolist()) <= got and len(got) >= k
        if kdist[i, -2] < r[i] * (1 - 1e-9):
            rp, idx, _ = oracle_mod.nwr(x, x, float(r[i]) * (1 - 1e-9), exclude_self=True,
                                        rows=[i])
            assert len(idx) == k - 1


def test_nwr_invariances(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((300, 6)).astype(np.float32)
    rp, idx, dist = oracle_mod.nwr(x, x, 2.0)
    perm = rng.permutation(len(x))
    rp2, idx2, dist2 = oracle_mod.nwr(x[perm], x[perm], 2.0)
    inv = np.argsort(perm)
    for i in range(len(x)):
        a = sorted(perm[idx2[rp2[inv[i]]:rp2[inv[i] + 1]]].tolist())
        assert a == idx[rp[i]:rp[i + 1]].tolist()
    rp3, idx3, dist3 = oracle_mod.nwr(x * 8, x * 8, 16.0)  # power-of-two scaling is exact
    np.testing.assert_array_equal(rp3, rp)
    np.testing.assert_array_equal(idx3, idx)
    np.testing.assert_array_equal(dist3, dist * 8)


def test_nwr_rejects_bad_arguments(oracle_mod):
    x = np.zeros((4, 2), np.float32)
    for phi in (-1.0, float("nan")):
        with pytest.raises(ValueError):
            oracle_mod.nwr(x, x, phi)


# ---------------------------------------------------------------------------
# kNN score variants (Table 1's kNN detector; Angiulli and Pizzuti's weight is
# the sum) and the kNN classifier's vote (Appendix B).
# ---------------------------------------------------------------------------

def _score_fixture():
    out = {}
    with open(os.path.join(os.path.dirname(__file__), "golden", "line10_scores.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, name, *vals = line.split()
            out[(int(k), name)] = [float(Fraction(v)) for v in vals]
    return out


@pytest.mark.parametrize("k", [2, 3])
@pytest.mark.parametrize("method", ["mean", "median", "sum"])
def test_score_variants_line_golden(oracle_mod, k, method):
    x = workloads.line(10, 1)
    _, dist = oracle_mod.knn_self(x, k)
    got = oracle_mod.knn_score(dist, method)
    np.testing.assert_allclose(got, _score_fixture()[(k, method)], rtol=1e-15, atol=0)
    np.testing.assert_array_equal(oracle_mod.knn_score(dist, "kth"), dist[:, -1])


def test_score_variants_lattice_closed_forms(oracle_mod):
    # 9 x 9 lattice, k = 4: interior points have four neighbours at 1; a
    # border point that is not a corner has three at 1 and a diagonal at
    # sqrt 2; a corner has two at 1, one at sqrt 2 and one at 2.
    x = workloads.lattice(9, 2)
    _, dist = oracle_mod.knn_self(x, 4)
    r2 = math.sqrt(2.0)
    want = {"interior": (1.0, 1.0, 4.0), "border": ((3 + r2) / 4, 1.0, 3 + r2),
            "corner": ((4 + r2) / 4, (1 + r2) / 2, 4 + r2)}
    scores = {m: oracle_mod.knn_score(dist, m) for m in ("mean", "median", "sum")}
    for i, (r, c) in enumerate(x.astype(int).tolist()):
        on_edge = (r in (0, 8)) + (c in (0, 8))
        kind = "corner" if on_edge == 2 else ("border" if on_edge == 1 else "interior")
        for m, v in zip(("mean", "median", "sum"), want[kind]):
            assert abs(scores[m][i] - v) <= 1e-15 * v, (i, kind, m, scores[m][i], v)


def test_vote_hand_examples(oracle_mod):
    # References at 0..9 on a line with labels 0,0,0,1,1,1,1,2,2,2.
    xr = workloads.line(10, 1)
    labels = np.array([0, 0, 0, 1, 1, 1, 1, 2, 2, 2], np.int32)
    xq = np.array([[2.6], [2.4], [6.6], [8.9]], np.float32)
    idx3, _ = oracle_mod.knn(xq, xr, 3)
    assert idx3.tolist() == [[3, 2, 4], [2, 3, 1], [7, 6, 8], [9, 8, 7]]
    assert oracle_mod.knn_vote(idx3, labels, 3).tolist() == [1, 0, 2, 2]
    idx2, _ = oracle_mod.knn(xq, xr, 2)
    # k = 2 near a class boundary: one vote each, the smaller label wins
    assert oracle_mod.knn_vote(idx2, labels, 3).tolist() == [0, 0, 1, 2]


def test_vote_matches_counting_by_hand(oracle_mod):
    rng = np.random.default_rng(8)
    idx = rng.integers(0, 50, (200, 7))
    labels = rng.integers(0, 4, 50).astype(np.int32)
    got = oracle_mod.knn_vote(idx, labels, 4)
    for r in range(len(idx)):
        votes = {}
        for j in idx[r]:
            votes[int(labels[j])] = votes.get(int(labels[j]), 0) + 1
        top = max(votes.values())
        assert got[r] == min(c for c, n in votes.items() if n == top)


# ---------------------------------------------------------------------------
# ABOD as the paper builds it (Section 4.3): kNN, then the mean cosine
# similarity of the difference vectors to each pair of neighbours.
# ---------------------------------------------------------------------------

def test_abod_line_closed_forms(oracle_mod):
    # k = 2: an interior point has neighbours on both sides (cosine -1); an
    # end point has both on one side (cosine 1).
    x = workloads.line(10, 1)
    idx, _ = oracle_mod.knn_self(x, 2)
    np.testing.assert_array_equal(oracle_mod.abod(x, idx), [1, -1, -1, -1, -1, -1, -1, -1, -1, 1])
    # k = 3: the ends see all three neighbours on one side; every other point
    # has two on one side and one on the other: cosines (-1, -1, 1) -> -1/3.
    idx, _ = oracle_mod.knn_self(x, 3)
    np.testing.assert_allclose(oracle_mod.abod(x, idx), [1] + [-1 / 3] * 8 + [1], rtol=1e-15)


def test_abod_lattice_closed_forms(oracle_mod):
    x = workloads.lattice(9, 2)
    idx, _ = oracle_mod.knn_self(x, 4)
    s = oracle_mod.abod(x, idx)
    # interior: four axis neighbours, 2 opposite pairs (-1) and 4 orthogonal (0)
    # corner (0, 0): neighbours (0,1), (1,0), (1,1), (0,2) (the lower index of the
    # tie at distance 2): cosines 0, 1/sqrt2, 1, 1/sqrt2, 0, 1/sqrt2
    r2 = math.sqrt(2.0)
    coords = x.astype(int).tolist()
    for i, (r, c) in enumerate(coords):
        if 1 <= r <= 7 and 1 <= c <= 7:
            assert abs(s[i] + 1 / 3) <= 1e-15
    assert abs(s[0] - (1 + 3 / r2) / 6) <= 1e-15


def test_abod_invariances_and_duplicates(oracle_mod):
    rng = np.random.default_rng(12)
    x = rng.standard_normal((120, 5)).astype(np.float32)
    idx, _ = oracle_mod.knn_self(x, 6)
    s = oracle_mod.abod(x, idx)
    # power-of-two scaling is exact and leaves every cosine unchanged; a row
    # permutation permutes the scores
    idx2, _ = oracle_mod.knn_self(x * 4, 6)
    np.testing.assert_array_equal(idx2, idx)
    np.testing.assert_allclose(oracle_mod.abod(x * 4, idx2), s, rtol=0, atol=1e-14)
    perm = rng.permutation(len(x))
    idx3, _ = oracle_mod.knn_self(x[perm], 6)
    np.testing.assert_allclose(oracle_mod.abod(x[perm], idx3), s[perm], rtol=0, atol=1e-14)
    assert np.all(np.abs(s) <= 1)
    # a duplicate neighbour (zero-length difference) is left out of the pairs
    xd = np.array([[0, 0], [0, 0], [1, 0], [-1, 0]], np.float32)
    idx, _ = oracle_mod.knn_self(xd, 3)
    assert idx[0].tolist() == [1, 2, 3]
    assert oracle_mod.abod(xd, idx)[0] == -1.0  # only the pair (2, 3) counts


# ---------------------------------------------------------------------------
# COF (Tang et al.; Table 1): set-based nearest path and average chaining
# distance from the kNN lists.
# ---------------------------------------------------------------------------

def _cof_fixture():
    out = {}
    with open(os.path.join(os.path.dirname(__file__), "golden", "cof_gaps.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, *vals = line.split()
            out[name] = [float(Fraction(v)) for v in vals]
    return out


def test_cof_golden_gaps(oracle_mod):
    fx = _cof_fixture()
    x = np.array(fx["x"], np.float32).reshape(-1, 1)
    idx, _ = oracle_mod.knn_self(x, 2)
    assert idx.tolist() == [[1, 2], [0, 2], [1, 0], [2, 4], [3, 2]]
    cof, ac = oracle_mod.cof(x, idx)
    np.testing.assert_allclose(ac, fx["ac"], rtol=1e-15)
    np.testing.assert_allclose(cof, fx["cof"], rtol=1e-9)


def test_cof_uniform_spacing_is_one(oracle_mod):
    # Every step of every path costs 1 on an evenly spaced line and on the
    # lattice interior, so ac = 1 (the weights sum to 1) and COF = 1.
    for x, k in ((workloads.line(10, 1), 2), (workloads.line(10, 1), 3),
                 (workloads.lattice(9, 2), 4)):
        idx, _ = oracle_mod.knn_self(x, k)
        cof, ac = oracle_mod.cof(x, idx)
        np.testing.assert_allclose(ac, 1.0, rtol=1e-15)
        np.testing.assert_allclose(cof, 1.0, rtol=1e-9)


def test_cof_scaling_and_duplicates(oracle_mod):
    rng = np.random.default_rng(14)
    x = rng.standard_normal((150, 4)).astype(np.float32)
    idx, _ = oracle_mod.knn_self(x, 5)
    cof, ac = oracle_mod.cof(x, idx)
    cof8, ac8 = oracle_mod.cof(x * 8, idx)  # distances scale exactly, ratios do not move
    np.testing.assert_allclose(ac8, 8 * ac, rtol=1e-15)
    np.testing.assert_allclose(cof8, cof, rtol=1e-9)
    assert np.all(cof > 0)
    dup = np.zeros((4, 2), np.float32)
    idx, _ = oracle_mod.knn_self(dup, 3)
    cof, ac = oracle_mod.cof(dup, idx)
    assert np.all(ac == 0) and np.all(cof == 1.0)


# ---------------------------------------------------------------------------
# LOCI (Papadimitriou et al.; Table 1): counting and sampling neighbourhoods at
# a ladder of radii, MDEF and its normalised deviation.
# ---------------------------------------------------------------------------

def _golden_value(v):
    if v.startswith("sqrt:"):
        return math.sqrt(float(Fraction(v[5:])))
    return float(Fraction(v))


def _loci_fixture():
    rows, scores = [], {}
    with open(os.path.join(os.path.dirname(__file__), "golden", "loci_line10.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            t = line.split()
            if t[0] == "score":
                scores[int(t[1])] = _golden_value(t[2])
            else:
                rows.append((int(t[0]), float(t[1]), int(t[2]), int(t[3]),
                             _golden_value(t[4]), _golden_value(t[5])))
    return rows, scores


def test_loci_golden_line(oracle_mod):
    rows, scores = _loci_fixture()
    radii = [1.0, 2.0, 4.0]
    r = oracle_mod.loci(workloads.line(10, 1), radii, alpha=0.5, n_min=1, k_sigma=3.0)
    for p, rad, na, nr, mdef, smdef in rows:
        li = radii.index(rad)
        for row in (p, 9 - p):  # the line is symmetric
            assert r["n_alpha"][row, li] == na and r["n_r"][row, li] == nr, (row, rad)
            assert abs(r["mdef"][row, li] - mdef) <= 1e-15 * max(1.0, abs(mdef)), (row, rad)
            assert abs(r["sigma_mdef"][row, li] - smdef) <= 1e-15, (row, rad)
    for p, v in scores.items():
        for row in (p, 9 - p):
            assert abs(r["score"][row] - v) <= 1e-14 * max(1.0, abs(v)), row
    assert not r["flag"].any()


def _loci_by_sets(x, radii, alpha, n_min, k_sigma):
    # The definition read directly: explicit neighbour sets per point and
    # radius, the sample mean and the population standard deviation of the
    # counting-neighbourhood sizes taken with the statistics module (two-pass),
    # squared distances as plain Python float sums over the columns.
    n = len(x)
    pts = [[float(v) for v in row] for row in x]

    def d2(p, q):
        s = 0.0
        for a, b in zip(pts[p], pts[q]):
            s = s + (a - b) * (a - b)
        return s

    dd = [[d2(p, q) for q in range(n)] for p in range(n)]
    out = []
    for p in range(n):
        per = []
        for r in radii:
            ra = alpha * r
            samp = [q for q in range(n) if dd[p][q] <= r * r]
            cnt = {q: sum(1 for o in range(n) if dd[q][o] <= ra * ra) for q in samp}
            vals = [cnt[q] for q in samp]
            nh = statistics.mean(vals)
            sd = statistics.pstdev(vals)
            na = sum(1 for o in range(n) if dd[p][o] <= ra * ra)
            per.append((na, len(samp), 1.0 - na / nh, sd / nh))
        counted = [v for v in per if v[1] >= n_min]
        ratios = [(v[2] / v[3]) if v[3] > 0 else 0.0 for v in counted]
        score = max(ratios) if ratios else 0.0
        flag = any(v[2] > k_sigma * v[3] for v in counted)
        out.append((per, score, flag))
    return out


@pytest.mark.parametrize("seed", [0, 1])
def test_loci_brute_force_sets(oracle_mod, seed):
    rng = np.random.default_rng(100 + seed)
    # two blobs and a few stragglers, with repeated points (ties on the radii)
    x = np.concatenate([rng.integers(0, 4, (20, 2)), rng.integers(8, 11, (14, 2)),
                        rng.integers(-9, 20, (6, 2))]).astype(np.float32)
    radii, alpha, n_min, ks = [1.0, 2.0, 3.0, 5.0, 8.0], 0.5, 4, 2.0
    r = oracle_mod.loci(x, radii, alpha, n_min, ks)
    ref = _loci_by_sets(x, radii, alpha, n_min, ks)
    for p, (per, score, flag) in enumerate(ref):
        for li, (na, nr, mdef, smdef) in enumerate(per):
            assert r["n_alpha"][p, li] == na and r["n_r"][p, li] == nr, (p, li)
            assert abs(r["mdef"][p, li] - mdef) <= 1e-12 * max(1.0, abs(mdef)), (p, li)
            assert abs(r["sigma_mdef"][p, li] - smdef) <= 1e-12, (p, li)
        assert abs(r["score"][p] - score) <= 1e-12 * max(1.0, abs(score)), p
        assert bool(r["flag"][p]) == flag, p
    assert r["flag"].any() and not r["flag"].all()


def test_loci_isolated_point_flagged(oracle_mod):
    # A 5 x 6 unit lattice (diameter sqrt(41)) and one point at (14, 15), at
    # least sqrt(200) from every lattice point and at most sqrt(421) < 21 from
    # any.  At r = 21 the lone point samples all 31 points; every counting
    # neighbourhood (alpha r = 10.5) of a lattice point holds the 30 lattice
    # points, the lone point's holds itself.
    lat = workloads.lattice(6, 2)[:30]
    x = np.concatenate([lat, [[14.0, 15.0]]]).astype(np.float32)
    r = oracle_mod.loci(x, [21.0], alpha=0.5, n_min=20, k_sigma=3.0)
    assert r["n_alpha"][30, 0] == 1 and r["n_r"][30, 0] == 31
    assert r["flag"][30] and not r["flag"][:30].any()
    # n_hat = (30 * 30 + 1) / 31, MDEF = 1 - 31 / 901 for the lone point
    assert abs(r["mdef"][30, 0] - (1.0 - 31.0 / 901.0)) < 1e-15


def test_loci_scaling_and_permutation(oracle_mod):
    rng = np.random.default_rng(7)
    x = rng.standard_normal((120, 3)).astype(np.float32)
    radii = [0.5, 0.8, 1.2, 1.9]
    r = oracle_mod.loci(x, radii, alpha=0.5, n_min=5, k_sigma=2.5)
    # power-of-two scaling of points and radii moves no squared distance or
    # threshold off its scaled value: every output is identical
    r4 = oracle_mod.loci(x * 4, [4 * v for v in radii], alpha=0.5, n_min=5, k_sigma=2.5)
    for key in r:
        np.testing.assert_array_equal(r4[key], r[key])
    perm = rng.permutation(120)
    rp = oracle_mod.loci(x[perm], radii, alpha=0.5, n_min=5, k_sigma=2.5)
    for key in r:
        np.testing.assert_array_equal(rp[key], r[key][perm])

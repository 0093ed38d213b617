"""Pins for the oracle's LOF on tie-inclusive k-distance neighbourhoods: hand-
derived values on integer points, a closed form with duplicate points, the
lattice's closed forms, agreement with the exactly-k LOF (pinned on its own)
where no distance ties, and invariances.  Never checked against itself or the
HIP path."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2110_14007_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sets():
    sets, cur = [], None
    with open(os.path.join(GOLDEN, "lof_ties.txt")) as f:
        for raw in f:
            raw = raw.strip()
            if not raw or raw.startswith("#"):
                continue
            t = raw.split()
            if t[0] == "set":
                cur = {"name": t[1], "k": int(t[2]), "x": [int(v) for v in t[3].split(",")]}
                sets.append(cur)
            else:
                cur[t[0]] = [Fraction(v) for v in t[1:]]
    return sets


@pytest.mark.parametrize("d", [1, 3])
@pytest.mark.parametrize("which", [0, 1])
def test_golden(oracle_mod, which, d):
    g = _sets()[which]
    x = np.zeros((len(g["x"]), d), np.float32)
    x[:, 0] = g["x"]
    lof, lrd, kdist, count = oracle_mod.lof_ties(x, g["k"])
    assert count.tolist() == [int(v) for v in g["count"]]
    np.testing.assert_array_equal(kdist, [float(v) for v in g["kdist"]])
    np.testing.assert_allclose(lrd, [float(v) for v in g["lrd"]], rtol=1e-9)
    np.testing.assert_allclose(lof, [float(v) for v in g["lof"]], rtol=1e-9)


def test_golden_differs_from_exactly_k(oracle_mod):
    # The fixture's tie at point 2 of line5 is what separates the two
    # neighbourhood rules: exactly k neighbours gives LOF(2) = 9/10.
    x = np.array([[0], [2], [3], [4], [8]], np.float32)
    idx, dist = oracle_mod.knn_self(x, 2)
    lof_k, _, _ = oracle_mod.lof(idx, dist)
    assert lof_k[1] == pytest.approx(0.9, rel=1e-9)
    assert oracle_mod.lof_ties(x, 2)[0][1] == pytest.approx(47 / 45, rel=1e-9)


def test_duplicates_closed_form(oracle_mod):
    # Points 0, 0, 1, 5 with k = 1.  The two zeros are each other's only
    # neighbour at distance 0, so kdist = 0 and lrd = 1 / (0 + 1e-10) = 1e10;
    # point 1 has both zeros tied at distance 1 (two neighbours, reach 1 each,
    # lrd = 1 / (1 + 1e-10)); point 5 has point 1 at distance 4 (reach
    # max(kdist(1) = 1, 4) = 4, lrd = 1 / (4 + 1e-10)).
    x = np.array([[0], [0], [1], [5]], np.float32)
    lof, lrd, kdist, count = oracle_mod.lof_ties(x, 1)
    assert count.tolist() == [1, 1, 2, 1]
    np.testing.assert_array_equal(kdist, [0.0, 0.0, 1.0, 4.0])
    np.testing.assert_allclose(lrd, [1e10, 1e10, 1 / (1 + 1e-10), 1 / (4 + 1e-10)], rtol=1e-14)
    np.testing.assert_allclose(lof, [1.0, 1.0, 1e10 * (1 + 1e-10), (4 + 1e-10) / (1 + 1e-10)],
                               rtol=1e-14)


def test_lattice_closed_forms(oracle_mod):
    # 9 x 9 integer grid, k = 5: a point off the edge has 4 neighbours at 1 and
    # 4 diagonal ones tied at sqrt 2, the 5th distance, so all 8 belong; every
    # reach distance is sqrt 2, and LOF = 1 wherever the neighbours' own
    # neighbourhoods are of that kind too (3 or more steps from the edge).
    side = 9
    x = workloads.lattice(side, 2)
    lof, lrd, kdist, count = oracle_mod.lof_ties(x, 5)
    c = x.astype(int)
    depth = np.minimum(c, side - 1 - c).min(axis=1)
    corner = (np.minimum(c, side - 1 - c) == 0).all(axis=1)
    assert np.all(count[depth >= 1] == 8)
    # Edge points: 3 at distance 1 and 2 at sqrt 2; corners: 2 at 1, 1 at
    # sqrt 2 and the two points 2 steps along the edges tied at 2.
    assert np.all(count[(depth == 0) & ~corner] == 5)
    assert np.all(count[corner] == 5)
    np.testing.assert_array_equal(kdist[~corner], math.sqrt(2.0))
    np.testing.assert_array_equal(kdist[corner], 2.0)
    np.testing.assert_allclose(lof[depth >= 3], 1.0, rtol=1e-9)
    np.testing.assert_allclose(lrd[depth >= 2], 1 / (math.sqrt(2.0) + 1e-10), rtol=1e-14)


@pytest.mark.parametrize("k", [1, 5, 12])
def test_equals_exactly_k_without_ties(oracle_mod, k):
    # Continuous data: no two distances from a point tie, so N_k(p) is the k
    # nearest and both rules give the same LOF.
    rng = np.random.default_rng(2024 + k)
    x = rng.standard_normal((300, 5)).astype(np.float32)
    lof, lrd, kdist, count = oracle_mod.lof_ties(x, k)
    assert np.all(count == k)
    idx, dist = oracle_mod.knn_self(x, k)
    lof_k, lrd_k, kdist_k = oracle_mod.lof(idx, dist)
    np.testing.assert_array_equal(kdist, kdist_k)
    np.testing.assert_allclose(lrd, lrd_k, rtol=1e-13)
    np.testing.assert_allclose(lof, lof_k, rtol=1e-13)


def test_invariances(oracle_mod):
    # Integer data with many ties: scaling by 4 and shifting by 16 (exact in
    # fp32 and fp64) keeps every neighbourhood, scales lrd by 1/4 and keeps
    # LOF (up to the 1e-10 guard); a permutation of the rows permutes the
    # outputs.
    rng = np.random.default_rng(77)
    x = rng.integers(0, 6, size=(120, 3)).astype(np.float32)
    lof, lrd, kdist, count = oracle_mod.lof_ties(x, 4)
    assert np.all(count >= 4) and np.any(count > 4)
    lof2, lrd2, kdist2, count2 = oracle_mod.lof_ties(4 * x + 16, 4)
    np.testing.assert_array_equal(count2, count)
    np.testing.assert_array_equal(kdist2, 4 * kdist)
    np.testing.assert_allclose(lof2, lof, rtol=1e-8)
    perm = rng.permutation(len(x))
    lof3, lrd3, kdist3, count3 = oracle_mod.lof_ties(x[perm], 4)
    np.testing.assert_array_equal(count3, count[perm])
    np.testing.assert_array_equal(kdist3, kdist[perm])
    np.testing.assert_allclose(lof3, lof[perm], rtol=1e-12)

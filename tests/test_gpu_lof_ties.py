"""GPU parity of LOF on tie-inclusive k-distance neighbourhoods (tod_lof_ties)
against the fp64 oracle.

Membership of a neighbourhood is decided in the definition's fp64 arithmetic
on both sides (columns in order, no fused multiply-add), so the sizes
|N_k(p)| must be identical on every row, ties included; LOF values agree
within the comparison rule's 1e-5 relative (fp32 output of fp64 sums taken
in a different order).  The data are chosen to be tie-heavy: integer points,
a lattice, repeated rows; continuous data check that the result is tod_lof's
wherever nothing ties.
"""
import os
import sys

import numpy as np
import pytest

from paper_2110_14007_amd import workloads
from tests.compare import compare_scores

pytestmark = pytest.mark.gpu

PRECS = ["fp16", "bf16"]
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2110_14007_amd import tod
    from oracle import oracle
    return torch, tod, oracle


def run(env, x, k, capacity=None, grow=True, **opt):
    torch, tod, _ = env
    a = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    st = tod.new_stats()
    lof, count = tod.tod_lof_ties(a, k, tod.options(**opt), capacity=capacity, grow=grow,
                                  stats=st)
    torch.cuda.synchronize()
    return lof.cpu().numpy(), count.cpu().numpy(), st.as_dict()


def check(env, x, k, **opt):
    _, _, oracle = env
    say("lof_ties n=%d d=%d k=%d %s" % (x.shape[0], x.shape[1], k, opt))
    lof, count, st = run(env, x, k, **opt)
    olof, _, _, ocount = oracle.lof_ties(x, k)
    np.testing.assert_array_equal(count, ocount)
    assert st["pairs_in_range"] == int(ocount.sum())
    compare_scores(lof, olof, what="lof")
    return lof, count, st


def _golden_sets():
    from fractions import Fraction
    sets, cur = [], None
    with open(os.path.join(GOLDEN, "lof_ties.txt")) as f:
        for raw in f:
            raw = raw.strip()
            if not raw or raw.startswith("#"):
                continue
            t = raw.split()
            if t[0] == "set":
                cur = {"k": int(t[2]), "x": [int(v) for v in t[3].split(",")]}
                sets.append(cur)
            else:
                cur[t[0]] = [Fraction(v) for v in t[1:]]
    return sets


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("which", [0, 1])
def test_golden(env, which, prec):
    g = _golden_sets()[which]
    x = np.zeros((len(g["x"]), 3), np.float32)
    x[:, 0] = g["x"]
    lof, count, _ = run(env, x, g["k"], precision=prec)
    assert count.tolist() == [int(v) for v in g["count"]]
    np.testing.assert_allclose(lof, [float(v) for v in g["lof"]], rtol=1e-6)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("n,d,k,hi", [(2000, 3, 4, 6), (2000, 3, 9, 6), (1500, 37, 5, 3),
                                      (2309, 8, 20, 4)])
def test_integer_points(env, n, d, k, hi, prec):
    rng = np.random.default_rng(9000 + n + d + k)
    x = rng.integers(0, hi, size=(n, d)).astype(np.float32)
    _, count, st = check(env, x, k, precision=prec)
    assert np.any(count > k)  # the data do tie
    assert st["pairs_candidate"] > 0  # so the range query ran


@pytest.mark.parametrize("k", [4, 5, 9, 12])
def test_lattice(env, k):
    x = workloads.lattice(41, 2)  # 1681 points, ties at every lattice distance
    check(env, x, k)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("k", [1, 2, 3, 6])
def test_repeated_rows(env, k, prec):
    # Every row three times: distance-0 neighbours, and ties at the k-distance
    # whenever it falls on a repeated point.
    rng = np.random.default_rng(31 + k)
    base = rng.standard_normal((700, 16)).astype(np.float32)
    x = np.repeat(base, 3, axis=0)
    check(env, x, k, precision=prec)


@pytest.mark.parametrize("prec", PRECS)
def test_continuous_equals_exactly_k(env, prec):
    # No ties: N_k(p) is the k nearest, and the scores are tod_lof's.
    torch, tod, _ = env
    x, _ = workloads.generate("C1", n=2500)
    lof, count, st = check(env, x, 10, precision=prec)
    assert np.all(count == 10)
    # Every 11th neighbour is farther than the 10th: the k-lists are the
    # neighbourhoods and the range query does not run.
    assert st["pairs_candidate"] == 0
    a = torch.from_numpy(x).cuda()
    lof_k, _ = tod.tod_lof(a, 10, tod.options(precision=prec))
    torch.cuda.synchronize()
    np.testing.assert_allclose(lof, lof_k.cpu().numpy(), rtol=1e-6)


def test_capacity_grows_and_reports(env):
    _, tod, _ = env
    rng = np.random.default_rng(5)
    x = rng.integers(0, 5, size=(1200, 3)).astype(np.float32)
    k = 4
    with pytest.raises(tod.TodError) as e:
        run(env, x, k, capacity=len(x) * k, grow=False)
    assert e.value.status == tod.TOD_ERR_CAPACITY
    _, _, _, ocount = env[2].lof_ties(x, k)
    lof, count, st = run(env, x, k, capacity=len(x) * k)  # grows to the reported total
    np.testing.assert_array_equal(count, ocount)
    assert st["pairs_in_range"] == int(ocount.sum())


def test_c2_full_size_matches_exactly_k(env):
    # C2 (n = 100,000, d = 32, k = 20, continuous): no distance ties, so every
    # neighbourhood holds exactly k points and the scores equal tod_lof's,
    # whose own parity with the oracle is checked on sampled rows elsewhere.
    torch, tod, _ = env
    w = workloads.WORKLOADS["C2"]
    x, _ = workloads.generate("C2")
    say("lof_ties C2 full size")
    lof, count, st = run(env, x, w.k)
    assert np.all(count == w.k)
    assert st["pairs_candidate"] == 0 and st["pairs_in_range"] == len(x) * w.k
    a = torch.from_numpy(x).cuda()
    lof_k, _ = tod.tod_lof(a, w.k)
    torch.cuda.synchronize()
    np.testing.assert_allclose(lof, lof_k.cpu().numpy(), rtol=1e-6)


@pytest.mark.parametrize("prec", PRECS)
def test_degenerate_sets(env, prec):
    # All points equal: every other point ties at k-distance 0, so each
    # neighbourhood holds all n - 1 others and LOF = 1 (lrd = 1e10 everywhere).
    x = np.full((50, 5), 3.25, np.float32)
    lof, count, _ = check(env, x, 3, precision=prec)
    assert np.all(count == 49)
    np.testing.assert_allclose(lof, 1.0, rtol=1e-6)
    # Two points, k = 1; and k = n - 1 (every neighbourhood is all the others).
    rng = np.random.default_rng(11)
    check(env, rng.standard_normal((2, 7)).astype(np.float32), 1, precision=prec)
    _, count, _ = check(env, rng.standard_normal((40, 9)).astype(np.float32), 39,
                        precision=prec)
    assert np.all(count == 39)

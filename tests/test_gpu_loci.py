"""GPU parity of LOCI (tod_loci) against the fp64 oracle.

Neighbourhood membership is exact on both sides (the same fp64 squared
distance, compared with the same fp64 thresholds), so the counts must be
identical, radii placed exactly on pair distances included.  The sums are
exact integers and the remaining steps are the same correctly rounded fp64
operations in the same order, so MDEF and sigma_MDEF are compared to 1e-12
relative (in practice they agree bit for bit) and the flags exactly.
"""
import sys

import numpy as np
import pytest

from paper_2110_14007_amd import workloads

pytestmark = pytest.mark.gpu


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


def run_loci(env, x, radii, alpha, n_min, k_sigma, capacity=None, **opt):
    torch, tod, _ = env
    xd = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    st = tod.new_stats()
    score, flag, ext = tod.tod_loci(xd, radii, alpha, n_min, k_sigma, tod.options(**opt),
                                    capacity=capacity, stats=st, return_all=True)
    torch.cuda.synchronize()
    out = {"score": score.cpu().numpy(), "flag": flag.cpu().numpy().astype(bool)}
    out.update({k: v.cpu().numpy() for k, v in ext.items()})
    return out, st.as_dict()


def check(env, x, radii, alpha=0.5, n_min=20, k_sigma=3.0, **opt):
    _, _, oracle = env
    say("loci n=%d d=%d radii=%s alpha=%g n_min=%d opts=%s" % (x.shape[0], x.shape[1],
                                                              list(radii), alpha, n_min, opt))
    g, st = run_loci(env, x, radii, alpha, n_min, k_sigma, **opt)
    o = oracle.loci(x, radii, alpha, n_min, k_sigma)
    np.testing.assert_array_equal(g["n_alpha"], o["n_alpha"])
    np.testing.assert_array_equal(g["n_r"], o["n_r"])
    np.testing.assert_allclose(g["mdef"], o["mdef"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g["sigma_mdef"], o["sigma_mdef"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g["score"], o["score"], rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(g["flag"], o["flag"])
    assert st["pairs_in_range"] == int(o["n_r"][:, -1].sum())
    return g, o, st


def test_line_golden_case(env):
    g, o, _ = check(env, workloads.line(10, 1), [1.0, 2.0, 4.0], alpha=0.5, n_min=1)
    assert abs(g["score"][0] - 1.75) < 1e-14 and not g["flag"].any()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_integer_blobs_with_ties(env, seed):
    # integer coordinates: many pair distances fall exactly on the radii
    rng = np.random.default_rng(500 + seed)
    x = np.concatenate([rng.integers(0, 6, (150, 2)), rng.integers(20, 24, (90, 2)),
                        rng.integers(-30, 50, (20, 2))]).astype(np.float32)
    radii = [1.0, 2.0, 3.0, 5.0, 8.0, 13.0]
    g, o, _ = check(env, x, radii, alpha=0.5, n_min=10, k_sigma=2.0)
    assert o["flag"].any()


@pytest.mark.parametrize("d,nl", [(16, 8), (5, 12), (3, 32)])
def test_gaussian_mixture(env, d, nl):
    # d = 5: rows that are not a multiple of four elements; nl > 8 and = 32:
    # the wider count-table layouts
    rng = np.random.default_rng(d * 100 + nl)
    n = 2500
    x = np.concatenate([rng.standard_normal((n - 100, d)),
                        rng.uniform(-6, 6, (100, d))]).astype(np.float32)
    typical = np.sqrt(2.0 * d)
    radii = list(np.geomspace(0.45 * typical, 1.1 * typical, nl))
    check(env, x, radii, alpha=0.5, n_min=20, k_sigma=3.0)


@pytest.mark.parametrize("opt", [dict(precision="bf16"), dict(force_fallback=True),
                                 dict(ref_splits=3), dict(margin_scale=50.0)])
def test_filter_options_do_not_change_results(env, opt):
    rng = np.random.default_rng(77)
    x = np.concatenate([rng.standard_normal((1200, 8)) * 0.5,
                        rng.standard_normal((800, 8)) + 3.0]).astype(np.float32)
    radii = [0.8, 1.1, 1.5, 2.0, 2.6]
    base, _ = run_loci(env, x, radii, 0.5, 15, 3.0)
    other, _ = run_loci(env, x, radii, 0.5, 15, 3.0, **opt)
    for key in base:
        np.testing.assert_array_equal(other[key], base[key])
    check(env, x, radii, alpha=0.5, n_min=15, k_sigma=3.0, **opt)


def test_degenerate_inputs(env):
    # one point: it is its own only neighbour, MDEF 0, no radius counts for n_min 2
    g, _, _ = check(env, np.zeros((1, 4), np.float32), [0.0, 1.0], alpha=0.5, n_min=2)
    assert g["score"][0] == 0.0 and not g["flag"][0]
    # all points equal: every neighbourhood is the whole set at every radius (r = 0 included)
    g, _, _ = check(env, np.ones((70, 3), np.float32), [0.0, 0.5], alpha=1.0, n_min=1)
    assert np.all(g["n_r"] == 70) and np.all(g["mdef"] == 0.0) and not g["flag"].any()
    # a single radius, alpha = 1 (counting = sampling neighbourhood)
    rng = np.random.default_rng(3)
    check(env, rng.standard_normal((400, 4)).astype(np.float32), [1.7], alpha=1.0, n_min=5)


def test_capacity_retry_and_error(env):
    torch, tod, _ = env
    rng = np.random.default_rng(5)
    x = rng.standard_normal((600, 4)).astype(np.float32)
    radii = [1.0, 2.0, 3.5]
    o = env[2].loci(x, radii, 0.5, 10, 3.0)
    need = int(o["n_r"][:, -1].sum())
    xd = torch.from_numpy(x).cuda()
    with pytest.raises(tod.TodError) as e:
        tod.tod_loci(xd, radii, 0.5, 10, 3.0, capacity=need - 1, grow=False)
    assert e.value.status == tod.TOD_ERR_CAPACITY
    st = tod.new_stats()
    score, flag = tod.tod_loci(xd, radii, 0.5, 10, 3.0, capacity=600, stats=st)  # grows once
    torch.cuda.synchronize()
    assert st.pairs_in_range == need
    np.testing.assert_allclose(score.cpu().numpy(), o["score"], rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(flag.cpu().numpy().astype(bool), o["flag"])


def test_full_size_workload_sampled(env):
    """The benchmark workload: exact counts of sampled rows from the oracle's
    neighbours within each radius; the neighbourhood sums of those rows from
    the GPU's own counting-neighbourhood table over the oracle's neighbour
    sets; properties of every row."""
    _, _, oracle = env
    w = workloads.WORKLOADS["L1"]
    x, _ = workloads.generate("L1")
    p = w.extra
    radii, alpha, n_min, ks = p["radii"], p["alpha"], p["n_min"], p["k_sigma"]
    g, st = run_loci(env, x, radii, alpha, n_min, ks)
    say("L1: pairs within the largest radius %d, stats %s" % (st["pairs_in_range"], st))
    n, nl = x.shape[0], len(radii)
    assert np.all(g["n_alpha"] >= 1) and np.all(g["n_r"] >= g["n_alpha"])
    assert np.all(np.diff(g["n_r"], axis=1) >= 0) and np.all(np.diff(g["n_alpha"], axis=1) >= 0)
    assert st["pairs_in_range"] == int(g["n_r"][:, -1].sum())
    rows = workloads.sample_rows("L1", count=48)
    for li, r in enumerate(radii):
        rp, idx, _ = oracle.nwr(x, x, r, rows=rows)
        np.testing.assert_array_equal(g["n_r"][rows, li], np.diff(rp))
        ra = float(np.float64(alpha) * np.float64(r))
        rpa, _, _ = oracle.nwr(x, x, ra, rows=rows)
        np.testing.assert_array_equal(g["n_alpha"][rows, li], np.diff(rpa))
        for t, pt in enumerate(rows):
            nb = idx[rp[t]:rp[t + 1]]
            vals = g["n_alpha"][nb, li].astype(np.int64)
            nr = float(len(nb))
            nhat = float(vals.sum()) / nr
            var = float((vals * vals).sum()) / nr - nhat * nhat
            var = max(var, 0.0)
            mdef = 1.0 - float(g["n_alpha"][pt, li]) / nhat
            smdef = np.sqrt(var) / nhat
            assert abs(g["mdef"][pt, li] - mdef) <= 1e-12 * max(1.0, abs(mdef)), (pt, li)
            assert abs(g["sigma_mdef"][pt, li] - smdef) <= 1e-12, (pt, li)
    counted = g["n_r"] >= n_min
    ratio = np.where(g["sigma_mdef"] > 0, g["mdef"] / np.where(g["sigma_mdef"] > 0,
                                                                g["sigma_mdef"], 1.0), 0.0)
    ref = np.where(counted.any(axis=1), np.where(counted, ratio, -np.inf).max(axis=1), 0.0)
    np.testing.assert_allclose(g["score"], ref, rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(g["flag"], (counted & (g["mdef"] > ks * g["sigma_mdef"])).any(1))
    say("L1: %d of %d points flagged" % (int(g["flag"].sum()), n))

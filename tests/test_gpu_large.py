"""GPU parity at the full workload sizes, in the launch configuration the
benchmark uses.  The oracle checks a seeded sample of rows one by one
(exact fp64 brute force against the whole reference set); every row is
checked for the properties that hold at any size; and the low-precision
filters are checked against the fp32 filter on every row (provable
quantization: the final answer does not depend on the filter)."""
import sys

import numpy as np
import pytest

from paper_2110_14007_amd import workloads
from tests.compare import compare_knn, compare_scores

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


def gpu_lists(env, x, k, lof, **opt):
    torch, tod, _ = env
    xd = torch.from_numpy(x).cuda()
    st = tod.new_stats()
    if lof:
        lofv, score, idx, dist = tod.tod_lof(xd, k, tod.options(**opt), stats=st,
                                             return_lists=True)
        lofv = lofv.cpu().numpy()
    else:
        score, idx, dist = tod.tod_knn_score(xd, k, tod.options(**opt), stats=st,
                                             return_lists=True)
        lofv = None
    torch.cuda.synchronize()
    out = (score.cpu().numpy(), idx.cpu().numpy(), dist.cpu().numpy(), lofv, st.as_dict())
    del xd, score, idx, dist
    torch.cuda.empty_cache()
    return out


def check_properties(x, k, score, idx, dist, lofv):
    n = x.shape[0]
    assert idx.shape == (n, k)
    assert np.all((idx >= 0) & (idx < n))
    assert not np.any(idx == np.arange(n)[:, None]), "self must be excluded"
    s = np.sort(idx, axis=1)
    assert not np.any(s[:, 1:] == s[:, :-1]), "neighbours must be distinct"
    assert np.all(np.diff(dist, axis=1) >= 0), "rows sorted by distance"
    np.testing.assert_array_equal(score, dist[:, -1])
    if lofv is not None:
        assert np.all(np.isfinite(lofv)) and np.all(lofv > 0)


def run_config(env, name, nrows=2048, lof_rows=0, cross_check=None, repeat=False):
    _, _, oracle = env
    w = workloads.WORKLOADS[name]
    x, _ = workloads.generate(name)
    say("%s: generated %s" % (name, x.shape))
    lof = w.lof or lof_rows > 0
    score, idx, dist, lofv, st = gpu_lists(env, x, w.k, lof, query_block=w.query_block)
    say("%s: gpu stats %s" % (name, st))
    check_properties(x, w.k, score, idx, dist, lofv)
    rows = workloads.sample_rows(name, count=nrows)
    oidx, odist = oracle.knn_self(x, w.k, rows=rows)
    n_exc, exc = compare_knn(x, x, rows, idx[rows], dist[rows], oidx, odist)
    compare_scores(score[rows], odist[:, -1], rows, exc, what="kNN score")
    say("%s: %d sampled rows match the oracle (%d excused near-ties)" % (name, len(rows), n_exc))
    if lof_rows:
        r = rows[:lof_rows]
        olof, _, _ = oracle.lof_rows(x, w.k, r)
        compare_scores(lofv[r], olof, what="LOF")
        say("%s: LOF of %d sampled rows matches the oracle" % (name, len(r)))
    if repeat:
        # The same call again: every output bit for bit, on every row.
        s2, i2, d2, l2, _ = gpu_lists(env, x, w.k, lof, query_block=w.query_block)
        np.testing.assert_array_equal(i2, idx)
        np.testing.assert_array_equal(d2, dist)
        np.testing.assert_array_equal(s2, score)
        if lof:
            np.testing.assert_array_equal(l2, lofv)
        # The filter's own lists, unverified (no_recheck keeps the shortlist's
        # first k in key order): two runs of the fused tile agree bit for bit.
        r1 = gpu_lists(env, x, w.k, False, query_block=w.query_block, no_recheck=True)
        r2 = gpu_lists(env, x, w.k, False, query_block=w.query_block, no_recheck=True)
        np.testing.assert_array_equal(r1[1], r2[1])
        np.testing.assert_array_equal(r1[2], r2[2])
        say("%s: two runs identical on every row (verified and unverified)" % name)
    if cross_check:
        s2, i2, d2, l2, st2 = gpu_lists(env, x, w.k, lof, query_block=w.query_block,
                                        precision=cross_check)
        say("%s: %s filter stats %s" % (name, cross_check, st2))
        np.testing.assert_array_equal(i2, idx)
        np.testing.assert_array_equal(d2, dist)
        if lof:
            np.testing.assert_array_equal(l2, lofv)
    return st


def test_C2_full_size(env):
    run_config(env, "C2", nrows=2048, lof_rows=64, cross_check="fp32")


def test_C3_full_size(env):
    run_config(env, "C3", nrows=2048, lof_rows=32, cross_check="fp32", repeat=True)


def test_C4_full_size(env):
    # the workload's bf16 filter against the library's default (fp16)
    st = run_config(env, "C4", nrows=2048, lof_rows=2, cross_check="bf16")
    assert st["precision"] == "fp16"


def test_C5_full_size(env):
    run_config(env, "C5", nrows=2048, lof_rows=32, cross_check="fp32", repeat=True)

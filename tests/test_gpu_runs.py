"""GPU parity of the two-run shortlist: K' = 128 on rows of 129..512
elements (a bf16 filter at k of 33..64) is built by the register-list tile as
two runs of 64 entries, one per piece of the scan order, and the recheck
merges them and bounds the excluded references by the smaller run end.
Every row is compared with the oracle; the outputs must not depend on how
the scan was cut (reference splits, query blocks, grouped order)."""
import sys

import numpy as np
import pytest

from tests.compare import compare_knn, compare_scores
from tests.test_gpu_shapes import lowrank

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


def run_lof(env, x, k, **opt):
    torch, tod, _ = env
    xd = torch.from_numpy(x).cuda()
    st = tod.new_stats()
    out = tod.tod_lof(xd, k, tod.options(**opt), stats=st, return_lists=True)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out], st.as_dict()


def check_rows(env, x, k, res):
    _, _, oracle = env
    lof, score, idx, dist = res
    oidx, odist = oracle.knn_self(x, k)
    olof, _, okd = oracle.lof(oidx, odist)
    rows = np.arange(len(x))
    n_exc, exc = compare_knn(x, x, rows, idx, dist, oidx, odist)
    compare_scores(score, okd, what="kNN score")
    touched = set(exc)
    for r in exc:
        touched.update(np.nonzero((oidx == r).any(axis=1))[0].tolist())
    compare_scores(lof, olof, rows, touched, what="LOF")
    return n_exc


@pytest.mark.parametrize("n,d,k", [(4000, 512, 50), (3100, 300, 40), (2600, 129, 33),
                                   (2300, 256, 64)])
def test_two_runs_match_oracle(env, n, d, k):
    x = lowrank(n, d, 8100 + d)
    res, st = run_lof(env, x, k, precision="bf16")
    say("runs", n, d, k, st)
    assert st["kprime"] == 128 and st["list_runs"] == 2
    check_rows(env, x, k, res)


def test_two_runs_independent_of_the_cut(env):
    """Splits (pieces = 2 S), query blocks and the grouped order change how
    the references are cut into runs, never the outputs."""
    x = lowrank(3500, 384, 8200)
    k = 48
    base, st0 = run_lof(env, x, k, precision="bf16")
    assert st0["list_runs"] == 2
    check_rows(env, x, k, base)
    for opt in (dict(ref_splits=1), dict(ref_splits=3), dict(query_block=1000),
                dict(query_block=640, ref_splits=2), dict(reorder=-1), dict(force_fallback=1),
                dict(margin_scale=1e6)):
        got, st = run_lof(env, x, k, precision="bf16", **opt)
        say("cut", opt, st["ref_splits"], st["blocks"], st["reordered"], st["rows_fallback"])
        assert st["list_runs"] == 2
        for u, v in zip(got, base):
            np.testing.assert_array_equal(u, v)


def test_two_runs_cross_sets(env):
    """Separate query and reference sets (no self pair), ragged sizes, and
    more neighbours than one run holds after the merge would need."""
    torch, tod, oracle = env
    xr = lowrank(5003, 257, 8300)
    xq = lowrank(777, 257, 8301)
    k = 60
    st = tod.new_stats()
    idx, dist = tod.tod_knn(torch.from_numpy(xq).cuda(), torch.from_numpy(xr).cuda(), k,
                            tod.options(precision="bf16"), stats=st)
    say("cross runs", st.as_dict())
    assert st.list_runs == 2 and st.kprime == 128
    oidx, odist = oracle.knn(xq, xr, k)
    compare_knn(xq, xr, np.arange(len(xq)), idx.cpu().numpy(), dist.cpu().numpy(), oidx, odist)


def test_few_references_per_run(env):
    """Fewer references than K' in each piece: runs that are not full
    exclude nothing, so the certificate holds whatever the keys."""
    x = lowrank(150, 300, 8400)
    k = 40
    res, st = run_lof(env, x, k, precision="bf16", ref_splits=4)
    say("short runs", st)
    assert st["list_runs"] == 2
    check_rows(env, x, k, res)

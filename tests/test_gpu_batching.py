"""GPU parity of automatic batching sized to the caller's memory: a workspace
smaller than tod_workspace_size() makes the planner cut the queries into more,
smaller blocks (down to 32 rows); the results must be bit-identical to the
one-block run and match the oracle."""
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


def smallest_workspace(tod, nq, nr, d, k, mode, opts):
    """Bisect the host planner for the smallest workspace it accepts."""
    lo, hi = 0, tod.tod_workspace_size(nq, nr, d, k, mode, opts)
    while hi - lo > 1:
        mid = (lo + hi) // 2
        try:
            tod.tod_plan_workspace(nq, nr, d, k, mid, mode, opts)
            hi = mid
        except tod.TodError:
            lo = mid
    return hi


@pytest.mark.parametrize("prec", ["fp16", "fp32"])
def test_lof_small_workspaces(env, prec):
    torch, tod, oracle = env
    x, _ = workloads.generate("C2", n=12000)
    n, d = x.shape
    k = 20
    opts = tod.options(precision=prec)
    xd = torch.from_numpy(x).cuda()
    base = [t.cpu().numpy() for t in tod.tod_lof(xd, k, opts, return_lists=True)]
    oidx, odist = oracle.knn_self(x, k)
    olof, _, okd = oracle.lof(oidx, odist)
    rows = np.arange(n)
    _, exc = compare_knn(x, x, rows, base[2], base[3], oidx, odist)
    compare_scores(base[1], okd, what="kNN score")
    touched = set(exc)
    for r in exc:
        touched.update(np.nonzero((oidx == r).any(axis=1))[0].tolist())
    compare_scores(base[0], olof, rows, touched, what="LOF")
    full = tod.tod_workspace_size(n, n, d, k, 1, opts)
    fplan = tod.tod_plan_workspace(n, n, d, k, full, 1, opts)
    least = smallest_workspace(tod, n, n, d, k, 1, opts)
    assert least < full
    for nbytes in (least, least + 40 * 32 * 8 * 64, (least + full) // 2):
        plan = tod.tod_plan_workspace(n, n, d, k, nbytes, 1, opts)
        ws = tod.FixedWorkspace(nbytes)
        st = tod.new_stats()
        got = [t.cpu().numpy() for t in tod.tod_lof(xd, k, opts, workspace=ws, stats=st,
                                                      return_lists=True)]
        say(prec, "workspace", nbytes, "of", full, "plan", plan, "blocks", st.blocks)
        assert st.blocks == plan["blocks"] and st.query_block == plan["query_block"]
        assert st.ref_splits == plan["ref_splits"]
        # a smaller workspace cuts the queries into more blocks or the
        # references into fewer splits; the smallest one leaves 32-row blocks
        assert st.blocks > 1 or st.ref_splits < fplan["ref_splits"]
        if nbytes == least:
            assert st.query_block == 32
        for u, v in zip(got, base):
            np.testing.assert_array_equal(u, v)
    with pytest.raises(tod.TodError) as e:
        tod.tod_lof(xd, k, opts, workspace=tod.FixedWorkspace(least - 256))
    assert e.value.status == tod.TOD_ERR_WORKSPACE


def test_knn_cross_small_workspace(env):
    torch, tod, oracle = env
    rng = np.random.default_rng(77)
    xr = rng.standard_normal((9000, 24)).astype(np.float32)
    xq = rng.standard_normal((1999, 24)).astype(np.float32)
    k = 9
    a, b = torch.from_numpy(xq).cuda(), torch.from_numpy(xr).cuda()
    opts = tod.options()
    idx0, dist0 = tod.tod_knn(a, b, k, opts)
    oidx, odist = oracle.knn(xq, xr, k)
    compare_knn(xq, xr, np.arange(len(xq)), idx0.cpu().numpy(), dist0.cpu().numpy(), oidx, odist)
    least = smallest_workspace(tod, len(xq), len(xr), 24, k, 0, opts)
    st = tod.new_stats()
    idx, dist = tod.tod_knn(a, b, k, opts, workspace=tod.FixedWorkspace(least + 1000), stats=st)
    say("cross: blocks", st.blocks, "query block", st.query_block)
    assert st.blocks > 1
    np.testing.assert_array_equal(idx.cpu().numpy(), idx0.cpu().numpy())
    np.testing.assert_array_equal(dist.cpu().numpy(), dist0.cpu().numpy())

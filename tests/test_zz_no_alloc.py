"""tod_knn_noalloc (the library's static scratch as the workspace) against
tod_knn with a workspace of its own: identical outputs on consecutive calls,
the later ones smaller (the scratch keeps the earlier call's contents), a
problem the planner must batch to fit the scratch, and a clear
TOD_ERR_WORKSPACE for one that cannot fit.  Also checked against the oracle
on the small calls."""
import sys

import numpy as np
import pytest

from tests.compare import compare_knn

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


def both(tod, torch, xq, xr, k, opts=None):
    a, b = torch.from_numpy(xq).cuda(), torch.from_numpy(xr).cuda()
    if xq is xr:
        b = a
    idx0, dist0 = tod.tod_knn(a, b, k, opts)
    st = tod.new_stats()
    idx1, dist1 = tod.tod_knn_noalloc(a, b, k, opts, stats=st)
    torch.cuda.synchronize()
    return (idx0.cpu().numpy(), dist0.cpu().numpy(), idx1.cpu().numpy(), dist1.cpu().numpy(), st)


def test_consecutive_calls_match_tod_knn(env):
    torch, tod, oracle = env
    rng = np.random.default_rng(4242)
    cases = [  # (nq, nr, d, k), later calls smaller
        (6000, 40000, 32, 20),
        (1000, 5000, 16, 10),
        (77, 300, 5, 3),
    ]
    for nq, nr, d, k in cases:
        say("noalloc case", nq, nr, d, k)
        xr = rng.standard_normal((nr, d)).astype(np.float32)
        xq = rng.standard_normal((nq, d)).astype(np.float32)
        i0, d0, i1, d1, st = both(tod, torch, xq, xr, k)
        np.testing.assert_array_equal(i1, i0)
        np.testing.assert_array_equal(d1, d0)
        assert st.blocks >= 1 and st.kprime >= k
        assert st.ms_total == 0.0  # no events inside the call
        rows = np.arange(nq) if nq <= 1000 else rng.choice(nq, 512, replace=False)
        oidx, odist = oracle.knn(xq, xr, k, rows=rows)
        compare_knn(xq, xr, rows, i1[rows], d1[rows], oidx, odist)


def test_batched_to_fit_scratch(env):
    torch, tod, oracle = env
    rng = np.random.default_rng(4343)
    n, d, k = 200_000, 32, 20
    x = rng.standard_normal((n, d)).astype(np.float32)
    # X against itself (the same layout with or without excluding the self pair)
    plan = tod.tod_plan_workspace(n, n, d, k, tod.NOALLOC_SCRATCH_BYTES, 0,
                                  tod.options(exclude_self=True))
    say("noalloc batched plan", plan)
    i0, d0, i1, d1, st = both(tod, torch, x, x, k)
    assert st.blocks == plan["blocks"] and st.blocks > 1
    np.testing.assert_array_equal(i1, i0)
    np.testing.assert_array_equal(d1, d0)
    # a smaller call right after the batched one
    i0, d0, i1, d1, st = both(tod, torch, x[:3000].copy(), x[:9000].copy(), 7)
    np.testing.assert_array_equal(i1, i0)
    np.testing.assert_array_equal(d1, d0)


def test_too_large_is_refused(env):
    torch, tod, _ = env
    n, d = 1_000_000, 64  # the quantised copy alone exceeds the scratch
    x = torch.zeros((n, d), dtype=torch.float32, device="cuda")
    with pytest.raises(tod.TodError) as e:
        tod.tod_knn_noalloc(x, x, 10)
    assert e.value.status == tod.TOD_ERR_WORKSPACE
    assert "static scratch" in str(e.value)
    # the library still works afterwards
    xs = torch.randn((500, 8), device="cuda")
    idx, dist = tod.tod_knn_noalloc(xs, xs, 4)
    idx0, dist0 = tod.tod_knn(xs, xs, 4)
    assert torch.equal(idx, idx0) and torch.equal(dist, dist0)

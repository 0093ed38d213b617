"""CPU checks of the batching planner (no GPU needed)."""
import pytest

from paper_2110_14007_amd import workloads


@pytest.fixture(scope="module")
def tod():
    from paper_2110_14007_amd import tod
    return tod


@pytest.mark.parametrize("name,prec,kp,blocks", [
    ("C1", "fp16", 32, 1), ("C2", "fp16", 32, 1), ("C3", "fp16", 32, 16), ("C4", "fp16", 64, 1),
    ("C5", "fp16", 16, 1)])
def test_plan_of_each_workload(tod, name, prec, kp, blocks):
    w = workloads.WORKLOADS[name]
    o = tod.options(exclude_self=True, query_block=w.query_block)
    p = tod.tod_plan(w.n, w.n, w.d, w.k, o)
    assert p["precision"] == prec
    assert p["kprime"] == kp and p["kprime"] >= w.k
    assert p["blocks"] == blocks
    if w.query_block:
        assert p["query_block"] == w.query_block
    assert 1 <= p["ref_splits"] <= 16


def test_explicit_options_respected(tod):
    o = tod.options(precision="bf16", shortlist=40, query_block=100, ref_splits=5)
    p = tod.tod_plan(1000, 3000, 20, 7, o)
    assert p["precision"] == "bf16"
    assert p["kprime"] == 64  # next power of two >= 40
    assert p["query_block"] == 128  # rounded up to a multiple of 32
    assert p["blocks"] == 8
    assert p["ref_splits"] == 5


@pytest.mark.parametrize("k", [1, 5, 20, 64, 100, 200, 256])
def test_kprime_covers_k(tod, k):
    for prec in ("fp32", "fp16", "bf16"):
        p = tod.tod_plan(5000, 5000, 16, k, tod.options(precision=prec))
        assert k <= p["kprime"] <= 256
        assert p["kprime"] & (p["kprime"] - 1) == 0


def test_workspace_grows_with_problem(tod):
    a = tod.tod_workspace_size(10000, 10000, 32, 10)
    b = tod.tod_workspace_size(20000, 20000, 32, 10)
    c = tod.tod_workspace_size(20000, 20000, 32, 10, mode=1)
    assert 0 < a < b
    assert c > 0
    assert tod.tod_workspace_size(10, 10, 4, 11) == 0  # k > nr
    assert tod.tod_workspace_size(10, 12, 4, 5, mode=1) == 0  # LOF needs nq == nr


@pytest.mark.parametrize("k,expect", [(5, 32), (10, 64), (20, 64), (50, 128), (200, 256)])
def test_bf16_shortlist_rule(tod, k, expect):
    # bf16 keeps k + max(24, k) candidates: at 2k about one row in ten of the
    # 4,000,000-point d = 8 workload (k = 5) fails the certificate.
    p = tod.tod_plan(5000, 5000, 16, k, tod.options(precision="bf16"))
    assert p["kprime"] == expect


def test_reorder_rule(tod):
    # X against X (tod_plan reads exclude_self as "the sets are one") through the
    # register-list kernel with one split and 4096+ references: grouped order.
    self_opts = dict(precision="fp16", exclude_self=True)
    assert tod.tod_plan(100000, 100000, 32, 20, tod.options(**self_opts))["reordered"]
    assert not tod.tod_plan(100000, 100000, 32, 20,
                            tod.options(reorder=-1, **self_opts))["reordered"]
    assert not tod.tod_plan(3000, 3000, 32, 20, tod.options(ref_splits=1, **self_opts))["reordered"]
    assert tod.tod_plan(3000, 3000, 32, 20,
                        tod.options(ref_splits=1, reorder=1, **self_opts))["reordered"]
    assert not tod.tod_plan(100000, 100000, 32, 20, tod.options(precision="fp16"))["reordered"]
    assert not tod.tod_plan(100000, 100000, 32, 20,
                            tod.options(precision="fp32", exclude_self=True))["reordered"]
    with pytest.raises(tod.TodError):
        tod.tod_plan(100, 100, 4, 3, tod.options(reorder=2))


def test_tail_region_in_workspace(tod):
    """The register-list tile with one reference split reserves the tail
    split's lists (query rows x 8 pieces, at most 2^18 lists of K' entries);
    tail_parts = 1 or a path without the tail split reserves none."""
    n, d, k = 100_000, 32, 20  # K' = 32, one split
    full = tod.tod_workspace_size(n, n, d, k, 1, tod.options(precision="fp16"))
    off = tod.tod_workspace_size(n, n, d, k, 1, tod.options(precision="fp16", tail_parts=1))
    lists = min(((n + 31) // 32 * 32) * 8, 1 << 18)
    assert full - off == lists * 32 * 8
    three = tod.tod_workspace_size(n, n, d, k, 1, tod.options(precision="fp16", tail_parts=3))
    assert three - off == min(((n + 31) // 32 * 32) * 3, 1 << 18) * 32 * 8
    small = 5000  # below the cap: the query rows times the pieces
    two = tod.tod_workspace_size(small, small, d, k, 1, tod.options(precision="fp16", tail_parts=2,
                                                                    ref_splits=1))
    none = tod.tod_workspace_size(small, small, d, k, 1, tod.options(precision="fp16",
                                                                     tail_parts=1, ref_splits=1))
    assert two - none == ((small + 31) // 32 * 32) * 2 * 32 * 8
    # fp32 filter (no register-list tile) and several reference splits: no tail region
    for o in (tod.options(precision="fp32"), tod.options(precision="fp32", tail_parts=1)):
        assert tod.tod_workspace_size(n, n, d, k, 1, o) == tod.tod_workspace_size(
            n, n, d, k, 1, tod.options(precision="fp32", tail_parts=1))
    assert tod.tod_workspace_size(n, n, d, k, 1, tod.options(precision="fp16", ref_splits=4)) == \
        tod.tod_workspace_size(n, n, d, k, 1, tod.options(precision="fp16", ref_splits=4,
                                                          tail_parts=1))


def test_workspace_sized_batching(tod):
    # Automatic batching sized to the caller's memory: smaller workspaces give
    # smaller query blocks (more blocks), down to one 32-row block.
    n, d, k = 100_000, 32, 20
    full = tod.tod_workspace_size(n, n, d, k, 1)
    big = tod.tod_plan_workspace(n, n, d, k, full, mode=1)
    assert big["blocks"] == 1 and big["query_block"] >= n
    prev = big
    sizes = [full * f // 100 for f in (60, 45, 35, 30)]
    for ws in sizes:
        p = tod.tod_plan_workspace(n, n, d, k, ws, mode=1)
        assert p["query_block"] % 32 == 0 and p["query_block"] <= prev["query_block"]
        assert p["blocks"] == -(-n // p["query_block"])
        prev = p
    assert prev["blocks"] > 1
    # the smallest workspace that still plans: bisect on the host planner
    lo, hi = 0, sizes[-1]
    while hi - lo > 1:
        mid = (lo + hi) // 2
        try:
            tod.tod_plan_workspace(n, n, d, k, mid, mode=1)
            hi = mid
        except tod.TodError as e:
            assert e.status == tod.TOD_ERR_WORKSPACE
            lo = mid
    p = tod.tod_plan_workspace(n, n, d, k, hi, mode=1)
    assert p["query_block"] == 32 and p["ref_splits"] == 1
    with pytest.raises(tod.TodError) as e:
        tod.tod_plan_workspace(n, n, d, k, hi - 1, mode=1)
    assert "32-row" in str(e.value)
    # a caller-fixed block is never re-planned
    with pytest.raises(tod.TodError):
        tod.tod_plan_workspace(n, n, d, k, sizes[0], mode=1, opts=tod.options(query_block=n))


@pytest.mark.parametrize("prec", ["fp16", "fp32", "bf16"])
@pytest.mark.parametrize("mode,nq,nr", [(1, 12000, 12000), (0, 1999, 9000), (1, 100_000, 100_000)])
def test_workspace_sweep_monotone(tod, prec, mode, nq, nr):
    # Every workspace size either plans or is refused as too small (never an
    # internal error), acceptance is monotone in the size, and a plan always
    # covers every query row.  Shrinking the reference splits of a self query
    # can switch the grouped scan order on, whose buffers the fitted layout
    # must then hold.
    d, k = 32, 20
    opts = tod.options(precision=prec)
    full = tod.tod_workspace_size(nq, nr, d, k, mode, opts)
    accepted = False
    for i in range(1, 161):
        ws = full * i // 160
        try:
            p = tod.tod_plan_workspace(nq, nr, d, k, ws, mode=mode, opts=opts)
        except tod.TodError as e:
            assert e.status == tod.TOD_ERR_WORKSPACE, str(e)
            assert not accepted, "refused %d bytes after accepting less" % ws
            continue
        accepted = True
        assert p["blocks"] * p["query_block"] >= nq
        assert p["blocks"] == -(-nq // p["query_block"])
        assert p["query_block"] % 32 == 0 or p["blocks"] == 1
    assert accepted

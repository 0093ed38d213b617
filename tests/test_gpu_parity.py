"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small cases are compared element by element on every row; integer-valued
pins allow no excused ties.  All inputs come from the seeded generators.
"""
import sys

import numpy as np
import pytest

from paper_2110_14007_amd import workloads
from tests.compare import compare_knn, compare_scores

pytestmark = pytest.mark.gpu

PRECS = ["fp32", "fp16", "bf16"]


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
    lof, score, idx, dist = tod.tod_lof(xd, k, tod.options(**opt), stats=st, return_lists=True)
    torch.cuda.synchronize()
    return (lof.cpu().numpy(), score.cpu().numpy(), idx.cpu().numpy(), dist.cpu().numpy(),
            st.as_dict())


def run_knn(env, xq, xr, k, **opt):
    torch, tod, _ = env
    a = torch.from_numpy(xq).cuda()
    b = a if xr is xq else torch.from_numpy(xr).cuda()
    st = tod.new_stats()
    idx, dist = tod.tod_knn(a, b, k, tod.options(**opt), stats=st)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), dist.cpu().numpy(), st.as_dict()


def check_full_lof(env, x, k, allow_ties=True, **opt):
    _, _, oracle = env
    lof, score, idx, dist, st = run_lof(env, x, k, **opt)
    oidx, odist = oracle.knn_self(x, k)
    olof, _, okd = oracle.lof(oidx, odist)
    rows = np.arange(len(x))
    n_exc, exc = compare_knn(x, x, rows, idx, dist, oidx, odist, allow_ties=allow_ties)
    compare_scores(score, okd, what="kNN score")
    # LOF rows touched by an excused tie (their own list or a neighbour's) are
    # excused too.
    touched = set(exc)
    for r in exc:
        touched.update(np.nonzero((oidx == r).any(axis=1))[0].tolist())
    compare_scores(lof, olof, rows, touched, what="LOF")
    return st, n_exc


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("k,d", [(2, 1), (3, 1), (3, 4)])
def test_line_pin(env, prec, k, d):
    say("line pin", prec, k, d)
    x = workloads.line(10, d)
    st, _ = check_full_lof(env, x, k, allow_ties=False, precision=prec)
    assert st["rows_certified"] + st["rows_fallback"] == 10


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("k", [4, 5, 8])
def test_lattice_pin(env, prec, k):
    say("lattice pin", prec, k)
    x = workloads.lattice(9, 2)
    check_full_lof(env, x, k, allow_ties=False, precision=prec)


def _tiny(case):
    rng = np.random.default_rng(4242 + case)
    n = int(rng.integers(2, 51))
    d = int(rng.choice([1, 2, 3, 5, 8, 17]))
    if case % 3 == 1:
        x = rng.integers(-3, 4, (n, d)).astype(np.float32)
    else:
        x = (rng.standard_normal((n, d)) * 10.0 ** rng.integers(-2, 3)).astype(np.float32)
    k = int(rng.integers(1, n))
    return x, k


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("case", range(12))
def test_tiny_exhaustive(env, prec, case):
    x, k = _tiny(case)
    say("tiny", prec, case, x.shape, k)
    check_full_lof(env, x, k, allow_ties=(case % 3 != 1), precision=prec)


@pytest.mark.parametrize("prec", PRECS)
def test_C1_full(env, prec):
    x, y = workloads.generate("C1")
    say("C1 full", prec)
    st, n_exc = check_full_lof(env, x, 10, precision=prec)
    say("stats", st, "excused", n_exc)


@pytest.mark.parametrize("prec", PRECS)
def test_cross_sets(env, prec):
    _, _, oracle = env
    rng = np.random.default_rng(17)
    xr = rng.standard_normal((3001, 37)).astype(np.float32)
    xq = rng.standard_normal((777, 37)).astype(np.float32)
    say("cross", prec)
    idx, dist, st = run_knn(env, xq, xr, 7, precision=prec)
    oidx, odist = oracle.knn(xq, xr, 7)
    compare_knn(xq, xr, np.arange(len(xq)), idx, dist, oidx, odist)


@pytest.mark.parametrize("prec", ["fp16", "bf16"])
@pytest.mark.parametrize("n,d,k", [(1000, 300, 5), (2500, 512, 20), (1777, 512, 50),
                                   (700, 257, 12)])
def test_wide_rows(env, prec, n, d, k):
    """Rows of 257..512 elements (the directly staged and the register-staged
    wide kernels, lists of 16, 32 and 64), ragged row counts, every row."""
    x, _ = workloads.generate("C4", n=n)
    x = np.ascontiguousarray(x[:, :d])
    say("wide rows", prec, n, d, k)
    st, n_exc = check_full_lof(env, x, k, precision=prec)
    say("stats", st, "excused", n_exc)


@pytest.mark.parametrize("prec", ["fp16", "bf16"])
def test_wide_rows_cross_and_splits(env, prec):
    _, _, oracle = env
    rng = np.random.default_rng(23)
    xr = rng.standard_normal((4001, 512)).astype(np.float32)
    xq = rng.standard_normal((333, 512)).astype(np.float32)
    for kw in (dict(), dict(ref_splits=3), dict(query_block=96)):
        say("wide cross", prec, kw)
        idx, dist, st = run_knn(env, xq, xr, 9, precision=prec, **kw)
        oidx, odist = oracle.knn(xq, xr, 9)
        compare_knn(xq, xr, np.arange(len(xq)), idx, dist, oidx, odist)


@pytest.mark.parametrize("prec", PRECS)
def test_C2_reduced_full(env, prec):
    x, _ = workloads.generate("C2", n=20000)
    say("C2 n=20000", prec)
    st, n_exc = check_full_lof(env, x, 20, precision=prec)
    say("stats", st, "excused", n_exc)


def test_precisions_agree_and_batching_invariant(env):
    # Provable quantization: the fp16 / bf16 shortlists and the fp32 one give
    # the same exact answer; so do other batchings and the forced fallback.
    x, _ = workloads.generate("C2", n=6000)
    say("invariance C2 n=6000")
    base = run_lof(env, x, 20, precision="fp32")
    variants = [dict(precision="fp16"), dict(precision="bf16"),
                dict(precision="fp16", query_block=64, ref_splits=7),
                dict(precision="fp32", query_block=1000, ref_splits=3),
                dict(precision="bf16", force_fallback=True),
                dict(precision="fp16", shortlist=20),
                dict(precision="fp16", margin_scale=1e6)]
    for v in variants:
        got = run_lof(env, x, 20, **v)
        say("variant", v, got[4])
        np.testing.assert_array_equal(got[2], base[2])
        np.testing.assert_array_equal(got[3], base[3])
        np.testing.assert_array_equal(got[0], base[0])
        np.testing.assert_array_equal(got[1], base[1])
    ff = run_lof(env, x, 20, precision="fp32", force_fallback=True)[4]
    assert ff["rows_fallback"] == len(x)


def test_deterministic(env):
    x, _ = workloads.generate("C1")
    a = run_lof(env, x, 10, precision="fp16")
    b = run_lof(env, x, 10, precision="fp16")
    for u, v in zip(a[:4], b[:4]):
        np.testing.assert_array_equal(u, v)


def test_no_recheck_changes_answers(env):
    # Without verification the fp16 shortlist order is returned as is; on
    # clustered data some neighbour lists change, which is what the exact
    # recheck prevents.
    x, _ = workloads.generate("C3", n=20000)
    say("no_recheck C3 n=20000")
    ref = run_lof(env, x, 10, precision="fp16")
    raw = run_lof(env, x, 10, precision="fp16", no_recheck=True)
    assert (raw[2] != ref[2]).any()


def test_nonfinite_rejected(env):
    torch, tod, _ = env
    x, _ = workloads.generate("C1", n=500)
    x = x.copy()
    x[17, 3] = np.nan
    with pytest.raises(tod.TodError) as e:
        tod.tod_lof(torch.from_numpy(x).cuda(), 5)
    assert e.value.status == tod.TOD_ERR_NONFINITE


def test_duplicates_and_minimal_sizes(env):
    _, _, oracle = env
    x = np.array([[1, 2], [1, 2], [1, 2], [3, 3], [0, 5]], np.float32)
    for prec in PRECS:
        check_full_lof(env, x, 2, allow_ties=False, precision=prec)
        check_full_lof(env, x, 4, allow_ties=False, precision=prec)
    x2 = np.array([[0.5], [2.0]], np.float32)
    for prec in PRECS:
        idx, dist, _ = run_knn(env, x2, x2, 2, precision=prec)
        assert idx.tolist() == [[0, 1], [1, 0]]
        np.testing.assert_array_equal(dist, [[0, 1.5], [0, 1.5]])


def test_large_values_and_offsets(env):
    # A common offset of 1e4 and a huge scale stress the centring, the
    # power-of-two scaling and the certificate.
    rng = np.random.default_rng(8)
    base = rng.standard_normal((3000, 24))
    for shift, scale in ((1e4, 1.0), (0.0, 1e30), (0.0, 1e-30), (-3e5, 1e-3)):
        x = (base * scale + shift).astype(np.float32)
        for prec in PRECS:
            say("offset/scale", shift, scale, prec)
            check_full_lof(env, x, 9, precision=prec)


@pytest.mark.parametrize("nq,nr,d,k", [(40, 40, 3, 7), (300, 300, 7, 9), (50, 3001, 37, 7),
                                       (1500, 1500, 5, 12), (7, 100, 2, 99)])
def test_forced_fallback_chunks(env, nq, nr, d, k):
    # Every row goes through the exact fallback scan.  With fewer failing rows
    # than the scan grid, each row's references are cut into chunks whose
    # sorted lists are merged; with more, one chunk is the whole row.
    _, _, oracle = env
    rng = np.random.default_rng(31 + nq + nr)
    xr = rng.integers(-4, 5, (nr, d)).astype(np.float32)  # many exact ties
    self_set = nq == nr
    xq = xr if self_set else rng.integers(-4, 5, (nq, d)).astype(np.float32)
    say("forced fallback", nq, nr, d, k)
    if self_set:
        check_full_lof(env, xr, k, allow_ties=False, force_fallback=True)
    else:
        idx, dist, st = run_knn(env, xq, xr, k, force_fallback=True)
        assert st["rows_fallback"] == nq
        oidx, odist = oracle.knn(xq, xr, k)
        compare_knn(xq, xr, np.arange(nq), idx, dist, oidx, odist, allow_ties=False)


# Grouped scan order (tod_options.reorder): the rows are partitioned and laid
# out group by group, each workgroup starts its scan at its own group, and the
# recheck maps positions back to input rows.  One reference split is forced:
# the order applies only then.
@pytest.mark.parametrize("case", ["line", "lattice", "ints", "dups", "C1", "tiny", "d11"])
def test_reorder_matches_oracle(env, case):
    rng = np.random.default_rng(41)
    if case == "line":
        x, k, ties = workloads.line(10, 4), 3, False
    elif case == "lattice":
        x, k, ties = workloads.lattice(9, 2), 5, False
    elif case == "ints":
        x, k, ties = rng.integers(-3, 4, (2500, 3)).astype(np.float32), 11, False
    elif case == "dups":
        base = rng.standard_normal((300, 6)).astype(np.float32)
        x, k, ties = np.concatenate([base, base[::3], base[::7]]), 6, False
    elif case == "C1":
        x, k, ties = workloads.generate("C1")[0], 10, True
    elif case == "d11":  # rows padded to 12 columns in the group assignment
        x, k, ties = rng.standard_normal((5000, 11)).astype(np.float32), 7, True
    else:
        x, k, ties = rng.standard_normal((70, 5)).astype(np.float32), 9, True
    say("reorder", case, x.shape, k)
    st, _ = check_full_lof(env, x, k, allow_ties=ties, precision="fp16", reorder=1, ref_splits=1)
    assert st["reordered"]


@pytest.mark.parametrize("prec", ["fp16", "bf16"])
def test_reorder_invariance(env, prec):
    x, _ = workloads.generate("C2", n=6000)
    on = run_lof(env, x, 20, precision=prec, reorder=1, ref_splits=1)
    off = run_lof(env, x, 20, precision=prec, reorder=-1, ref_splits=1)
    say("reorder invariance", prec, on[4], off[4])
    assert on[4]["reordered"] and not off[4]["reordered"]
    for u, v in zip(on[:4], off[:4]):
        np.testing.assert_array_equal(u, v)


def test_reorder_default(env):
    # The planner groups X-against-X scans of 4096+ references with one split.
    big, _ = workloads.generate("C2", n=5000)
    small, _ = workloads.generate("C2", n=3000)
    assert run_lof(env, big, 20, precision="fp16", ref_splits=1)[4]["reordered"]
    assert not run_lof(env, small, 20, precision="fp16", ref_splits=1)[4]["reordered"]
    xq = big[:500].copy()
    _, _, st = run_knn(env, xq, big, 5, precision="fp16", ref_splits=1)
    assert not st["reordered"]  # separate query set: input order


# Rows of at most 16 elements take one seed group per 8192 rows (32 groups at
# 300,000 rows, 64 at 600,000): the order must still change nothing, and
# sampled rows must match the oracle.
@pytest.mark.parametrize("n,d", [(300000, 8), (600000, 3)])
def test_reorder_many_groups(env, n, d):
    _, _, oracle = env
    rng = np.random.default_rng(n + d)
    x = rng.random((n, d), dtype=np.float64).astype(np.float32)
    say("reorder many groups", n, d)
    on = run_lof(env, x, 5, precision="fp16", reorder=1, ref_splits=1)
    off = run_lof(env, x, 5, precision="fp16", reorder=-1, ref_splits=1)
    assert on[4]["reordered"] and not off[4]["reordered"]
    for u, v in zip(on[:4], off[:4]):
        np.testing.assert_array_equal(u, v)
    rows = np.sort(rng.choice(n, 256, replace=False))
    oidx, odist = oracle.knn_self(x, 5, rows=rows)
    compare_knn(x, x, rows, on[2][rows], on[3][rows], oidx, odist)

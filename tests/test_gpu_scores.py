"""GPU parity of the kNN score variants (mean, median, sum), inductive
scoring of new points (tod_knn_decision) and the kNN classifier
(tod_knn_classify) against the oracle, through the C ABI."""
import sys

import numpy as np
import pytest

from paper_2110_14007_amd import workloads
from tests.compare import compare_knn, compare_scores

pytestmark = pytest.mark.gpu

METHODS = ["kth", "mean", "median", "sum"]


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


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("prec", ["fp32", "fp16", "bf16"])
def test_score_variants_pins(env, method, prec):
    torch, tod, oracle = env
    for x, k in ((workloads.line(10, 1), 2), (workloads.line(10, 1), 3),
                 (workloads.lattice(9, 2), 4), (workloads.lattice(9, 2), 8)):
        xd = torch.from_numpy(x).cuda()
        s = tod.tod_knn_score(xd, k, tod.options(precision=prec, score=method)).cpu().numpy()
        _, od = oracle.knn_self(x, k)
        np.testing.assert_allclose(s, oracle.knn_score(od, method), rtol=1e-6, atol=0)


@pytest.mark.parametrize("method", METHODS)
def test_score_variants_c2_reduced(env, method):
    torch, tod, oracle = env
    x, _ = workloads.generate("C2", n=20000)
    k = 20
    xd = torch.from_numpy(x).cuda()
    say("scores C2 n=20000", method)
    s, idx, dist = tod.tod_knn_score(xd, k, tod.options(score=method), return_lists=True)
    oidx, odist = oracle.knn_self(x, k)
    n_exc, exc = compare_knn(x, x, np.arange(len(x)), idx.cpu().numpy(), dist.cpu().numpy(),
                             oidx, odist)
    compare_scores(s.cpu().numpy(), oracle.knn_score(odist, method), np.arange(len(x)), set(exc),
                   what="kNN score (%s)" % method)
    # tod_lof reports the same score beside LOF
    lof, s2 = tod.tod_lof(xd, k, tod.options(score=method))
    np.testing.assert_array_equal(s2.cpu().numpy(), s.cpu().numpy())


@pytest.mark.parametrize("method", METHODS)
def test_decision_new_points(env, method):
    torch, tod, oracle = env
    x, _ = workloads.generate("C1")
    train, test = x[:1500], x[1500:]
    xr = torch.from_numpy(np.ascontiguousarray(train)).cuda()
    xq = torch.from_numpy(np.ascontiguousarray(test)).cuda()
    say("decision", method)
    s, idx, dist = tod.tod_knn_decision(xq, xr, 10, tod.options(score=method), return_lists=True)
    oidx, odist = oracle.knn(test, train, 10)
    n_exc, exc = compare_knn(test, train, np.arange(len(test)), idx.cpu().numpy(),
                             dist.cpu().numpy(), oidx, odist)
    compare_scores(s.cpu().numpy(), oracle.knn_score(odist, method), np.arange(len(test)),
                   set(exc), what="decision (%s)" % method)
    # the fitted points themselves: each is its own neighbour at distance 0
    s_self = tod.tod_knn_decision(xr, xr, 10, tod.options(score=method)).cpu().numpy()
    oidx, odist = oracle.knn(train, train, 10)
    assert np.all(odist[:, 0] == 0.0)
    compare_scores(s_self, oracle.knn_score(odist, method), what="decision on X (%s)" % method)


def test_decision_rejects_exclude_self(env):
    torch, tod, _ = env
    x = torch.from_numpy(workloads.line(10, 1)).cuda()
    with pytest.raises(tod.TodError) as e:
        tod.tod_knn_decision(x, x, 2, tod.options(exclude_self=True))
    assert e.value.status == tod.TOD_ERR_INVALID_ARG


def test_classifier_hand_example(env):
    torch, tod, _ = env
    xr = torch.from_numpy(workloads.line(10, 1)).cuda()
    labels = torch.tensor([0, 0, 0, 1, 1, 1, 1, 2, 2, 2], dtype=torch.int32, device="cuda")
    xq = torch.tensor([[2.6], [2.4], [6.6], [8.9]], dtype=torch.float32, device="cuda")
    assert tod.tod_knn_classify(xq, xr, labels, 3, 3).cpu().tolist() == [1, 0, 2, 2]
    assert tod.tod_knn_classify(xq, xr, labels, 2, 3).cpu().tolist() == [0, 0, 1, 2]


@pytest.mark.parametrize("prec", ["fp32", "fp16", "bf16"])
def test_classifier_against_oracle(env, prec):
    torch, tod, oracle = env
    rng = np.random.default_rng(31)
    centres = rng.uniform(-4, 4, (6, 12))
    lab = rng.integers(0, 6, 5000)
    train = (centres[lab] + rng.standard_normal((5000, 12))).astype(np.float32)
    lab_q = rng.integers(0, 6, 1300)
    test = (centres[lab_q] + rng.standard_normal((1300, 12))).astype(np.float32)
    labels = torch.from_numpy(lab.astype(np.int32)).cuda()
    xr, xq = torch.from_numpy(train).cuda(), torch.from_numpy(test).cuda()
    for k in (1, 7, 40):
        say("classifier", prec, k)
        pred = tod.tod_knn_classify(xq, xr, labels, k, 6, tod.options(precision=prec))
        oidx, odist = oracle.knn(test, train, k)
        want = oracle.knn_vote(oidx, lab, 6)
        # rows whose lists may legitimately differ (oracle near-ties) are excused
        idx, dist = tod.tod_knn(xq, xr, k, tod.options(precision=prec))
        _, exc = compare_knn(test, train, np.arange(len(test)), idx.cpu().numpy(),
                             dist.cpu().numpy(), oidx, odist)
        got = pred.cpu().numpy()
        bad = [r for r in np.nonzero(got != want)[0] if r not in exc]
        assert not bad, bad[:10]
    # X against itself, each point voting without itself
    self_pred = tod.tod_knn_classify(xr, xr, labels, 7, 6, tod.options(exclude_self=True))
    oidx, _ = oracle.knn_self(train, 7)
    np.testing.assert_array_equal(self_pred.cpu().numpy(), oracle.knn_vote(oidx, lab, 6))


def test_classifier_rejects_bad_labels(env):
    torch, tod, _ = env
    xr = torch.from_numpy(workloads.line(10, 1)).cuda()
    labels = torch.tensor([0, 0, 0, 1, 1, 5, 1, 2, 2, 2], dtype=torch.int32, device="cuda")
    with pytest.raises(tod.TodError) as e:
        tod.tod_knn_classify(xr, xr, labels, 3, 3)
    assert e.value.status == tod.TOD_ERR_INVALID_ARG


def _check_abod(env, x, k, allow_ties=True, **opt):
    torch, tod, oracle = env
    xd = torch.from_numpy(x).cuda()
    s, idx, dist = tod.tod_abod(xd, k, tod.options(**opt), return_lists=True)
    oidx, odist = oracle.knn_self(x, k)
    _, exc = compare_knn(x, x, np.arange(len(x)), idx.cpu().numpy(), dist.cpu().numpy(), oidx,
                         odist, allow_ties=allow_ties)
    want = oracle.abod(x, oidx)
    got = s.cpu().numpy().astype(np.float64)
    # a mean of cosines in [-1, 1], computed in fp64 and rounded once to fp32
    bad = [r for r in np.nonzero(np.abs(got - want) > 1e-6)[0] if r not in exc]
    assert not bad, (bad[:5], got[bad[:5]], want[bad[:5]])
    return got


@pytest.mark.parametrize("prec", ["fp32", "fp16", "bf16"])
def test_abod_pins(env, prec):
    x = workloads.line(10, 1)
    got = _check_abod(env, x, 2, allow_ties=False, precision=prec)
    np.testing.assert_array_equal(got, [1, -1, -1, -1, -1, -1, -1, -1, -1, 1])
    got = _check_abod(env, x, 3, allow_ties=False, precision=prec)
    np.testing.assert_allclose(got, [1] + [-1 / 3] * 8 + [1], atol=1e-7)
    _check_abod(env, workloads.lattice(9, 2), 4, allow_ties=False, precision=prec)
    xd = np.array([[0, 0], [0, 0], [1, 0], [-1, 0], [5, 5]], np.float32)
    _check_abod(env, xd, 3, allow_ties=False, precision=prec)


@pytest.mark.parametrize("n,d,k", [(2000, 16, 10), (3000, 32, 64), (1500, 200, 7),
                                   (777, 512, 2)])
def test_abod_against_oracle(env, n, d, k):
    name = "C1" if d == 16 else ("C2" if d == 32 else "C4")
    x, _ = workloads.generate(name, n=n)
    x = np.ascontiguousarray(x[:, :d])
    say("abod", n, d, k)
    _check_abod(env, x, k)


def test_abod_rejects_k(env):
    torch, tod, _ = env
    x = torch.from_numpy(workloads.line(100, 1)).cuda()
    for k, status in ((1, tod.TOD_ERR_INVALID_ARG), (65, tod.TOD_ERR_UNSUPPORTED)):
        with pytest.raises(tod.TodError) as e:
            tod.tod_abod(x, k)
        assert e.value.status == status


def _check_cof(env, x, k, allow_ties=True, **opt):
    torch, tod, oracle = env
    xd = torch.from_numpy(x).cuda()
    cof, score, idx, dist = tod.tod_cof(xd, k, tod.options(**opt), return_lists=True)
    oidx, odist = oracle.knn_self(x, k)
    _, exc = compare_knn(x, x, np.arange(len(x)), idx.cpu().numpy(), dist.cpu().numpy(), oidx,
                         odist, allow_ties=allow_ties)
    want, _ = oracle.cof(x, oidx)
    # rows touched by an excused tie (their own list or a neighbour's) are excused
    touched = set(exc)
    for r in exc:
        touched.update(np.nonzero((oidx == r).any(axis=1))[0].tolist())
    compare_scores(cof.cpu().numpy(), want, np.arange(len(x)), touched, what="COF")
    compare_scores(score.cpu().numpy(), odist[:, -1], np.arange(len(x)), set(exc),
                   what="kNN score beside COF")
    return cof.cpu().numpy()


@pytest.mark.parametrize("prec", ["fp32", "fp16", "bf16"])
def test_cof_pins(env, prec):
    x = np.array([[0], [1], [3], [6], [10]], np.float32)
    got = _check_cof(env, x, 2, allow_ties=False, precision=prec)
    np.testing.assert_allclose(got, [8 / 9, 8 / 9, 5 / 4, 5 / 4, 22 / 15], rtol=1e-6)
    for x, k in ((workloads.line(10, 1), 3), (workloads.lattice(9, 2), 4)):
        got = _check_cof(env, x, k, allow_ties=False, precision=prec)
        np.testing.assert_allclose(got, 1.0, rtol=1e-6)
    dup = np.zeros((6, 3), np.float32)
    np.testing.assert_array_equal(_check_cof(env, dup, 3, allow_ties=False, precision=prec), 1.0)


@pytest.mark.parametrize("n,d,k", [(2000, 16, 10), (1000, 32, 63), (800, 200, 5), (600, 512, 1)])
def test_cof_against_oracle(env, n, d, k):
    name = "C1" if d == 16 else ("C2" if d == 32 else "C4")
    x, _ = workloads.generate(name, n=n)
    x = np.ascontiguousarray(x[:, :d])
    say("cof", n, d, k)
    _check_cof(env, x, k)

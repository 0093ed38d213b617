"""GPU parity at the edges of the shapes the boundary accepts: rows of more
than 512 elements (up to the 4,096 limit; the paper's widest data set has
3,072 features) and the longest shortlists (K' = 256, k up to 256).  Every
row is compared with the oracle."""
import sys

import numpy as np
import pytest

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


def lowrank(n, d, seed):
    """Rank-16 Gaussian latent times a random projection, plus noise, and 1%
    full-rank outliers (the structure of wide tabular or image features)."""
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((16, d)) / 4.0
    x = rng.standard_normal((n, 16)) @ w + 0.1 * rng.standard_normal((n, d))
    out = rng.choice(n, max(1, n // 100), replace=False)
    x[out] = rng.standard_normal((len(out), d))
    return np.ascontiguousarray(x.astype(np.float32))


def run_score(env, x, k, **opt):
    torch, tod, _ = env
    xd = torch.from_numpy(x).cuda()
    st = tod.new_stats()
    lof, score, idx, dist = tod.tod_lof(xd, k, tod.options(**opt), stats=st, return_lists=True)
    torch.cuda.synchronize()
    return (lof.cpu().numpy(), score.cpu().numpy(), idx.cpu().numpy(), dist.cpu().numpy(),
            st.as_dict())


def check_all_rows(env, x, k, **opt):
    _, _, oracle = env
    lof, score, idx, dist, st = run_score(env, x, k, **opt)
    oidx, odist = oracle.knn_self(x, k)
    olof, _, okd = oracle.lof(oidx, odist)
    rows = np.arange(len(x))
    n_exc, exc = compare_knn(x, x, rows, idx, dist, oidx, odist)
    compare_scores(score, okd, what="kNN score")
    touched = set(exc)
    for r in exc:
        touched.update(np.nonzero((oidx == r).any(axis=1))[0].tolist())
    compare_scores(lof, olof, rows, touched, what="LOF")
    return st, n_exc


@pytest.mark.parametrize("prec", ["fp16", "bf16", "fp32"])
@pytest.mark.parametrize("n,d", [(2500, 513), (2200, 1000), (2000, 3072), (1500, 4096)])
def test_wide_beyond_512(env, prec, n, d):
    """Rows staged in column slabs (the LDS-list tile), ragged d and n."""
    x = lowrank(n, d, 7000 + d)
    say("wide", prec, n, d)
    st, n_exc = check_all_rows(env, x, 10, precision=prec)
    say("stats", st, "excused", n_exc)
    assert st["precision"] == prec


@pytest.mark.parametrize("prec", ["fp16", "bf16"])
@pytest.mark.parametrize("k", [128, 200, 256])
def test_longest_shortlists(env, prec, k):
    """k of 128..256 take K' = 256 (at k = 256 no margin is left, so every row
    goes through the exact fallback)."""
    x = lowrank(3000, 48, 7100 + k)
    say("long shortlist", prec, k)
    st, n_exc = check_all_rows(env, x, k, precision=prec)
    say("stats", st, "excused", n_exc)
    assert st["kprime"] == 256


def test_k256_fp32_and_cross(env):
    """k = 256 with an fp32 filter, and a separate query set at K' = 256."""
    _, _, oracle = env
    torch, tod, _ = env
    x = lowrank(2100, 20, 7400)
    st, _ = check_all_rows(env, x, 256, precision="fp32")
    assert st["kprime"] == 256
    xq = lowrank(333, 20, 7401)
    a, b = torch.from_numpy(xq).cuda(), torch.from_numpy(x).cuda()
    st = tod.new_stats()
    idx, dist = tod.tod_knn(a, b, 250, tod.options(precision="fp16"), stats=st)
    torch.cuda.synchronize()
    oidx, odist = oracle.knn(xq, x, 250)
    compare_knn(xq, x, np.arange(len(xq)), idx.cpu().numpy(), dist.cpu().numpy(), oidx, odist)
    assert st.kprime == 256

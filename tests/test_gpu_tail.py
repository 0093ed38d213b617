"""GPU parity of the tail split of the register-list tile.

When a query block's workgroups do not fill the GPU's last round, the tile
scans the references of the last round's workgroups in several pieces and
the recheck merges the pieces' lists.  The final neighbours are exact either
way, so every output must be identical with the split forced, chosen by the
planner and switched off, and match the oracle.
"""
import sys

import numpy as np
import pytest

from paper_2110_14007_amd import workloads
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


def run_lof(env, x, k, **opt):
    torch, tod, _ = env
    xd = torch.from_numpy(x).cuda()
    st = tod.new_stats()
    out = tod.tod_lof(xd, k, tod.options(**opt), stats=st, return_lists=True)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out], st.as_dict()


def run_knn(env, xq, xr, k, **opt):
    torch, tod, _ = env
    a = torch.from_numpy(xq).cuda()
    b = a if xr is xq else torch.from_numpy(xr).cuda()
    st = tod.new_stats()
    idx, dist = tod.tod_knn(a, b, k, tod.options(**opt), stats=st)
    torch.cuda.synchronize()
    return [idx.cpu().numpy(), dist.cpu().numpy()], st.as_dict()


@pytest.mark.parametrize("case", ["d32_lof", "d512_bf16", "d512_fp16", "d8_fold", "d64_fp16"])
def test_self_pieces_identical(env, case):
    """X against X (self excluded, grouped order): every output identical for
    2, 5 and 8 pieces, the planner's choice and no split; the 8-piece run
    against the oracle on every row."""
    _, _, oracle = env
    if case == "d32_lof":
        x, _ = workloads.generate("C2", n=9000)
        k, prec = 20, "fp16"
    elif case == "d512_bf16":
        x, _ = workloads.generate("C4", n=2600)
        k, prec = 20, "bf16"  # K' = 64
    elif case == "d512_fp16":
        x, _ = workloads.generate("C4", n=3100)
        k, prec = 20, "fp16"  # K' = 32: waves of 64 queries
    elif case == "d8_fold":
        x, _ = workloads.generate("C5", n=20000)
        k, prec = 5, "fp16"
    else:
        x, _ = workloads.generate("C3", n=7001)
        k, prec = 10, "fp16"
    base, st0 = run_lof(env, x, k, precision=prec, ref_splits=1, tail_parts=1)
    assert st0["tail_parts"] == 1 and st0["tail_rows"] == 0
    say(case, "no split", st0)
    for tp in (2, 5, 8, 0):
        got, st = run_lof(env, x, k, precision=prec, ref_splits=1, tail_parts=tp)
        say(case, "tail_parts", tp, "->", st["tail_parts"], "rows", st["tail_rows"],
            "launches", st["tile_launches"])
        if tp:
            assert st["tail_parts"] == tp and st["tail_rows"] > 0
        for u, v in zip(got, base):
            np.testing.assert_array_equal(u, v)
        if tp == 8:
            oidx, odist = oracle.knn_self(x, k)
            compare_knn(x, x, np.arange(len(x)), got[2], got[3], oidx, odist)


def test_cross_main_and_tail_launch(env):
    """More workgroups than the GPU holds at once: a full-round launch plus a
    tail launch in pieces, separate query and reference sets, ragged counts."""
    _, _, oracle = env
    rng = np.random.default_rng(41)
    xr = (rng.standard_normal((4133, 32)) * rng.uniform(0.5, 2.0, 32)).astype(np.float32)
    xq = (rng.standard_normal((70001, 32)) * rng.uniform(0.5, 2.0, 32)).astype(np.float32)
    k = 12
    base, st0 = run_knn(env, xq, xr, k, precision="fp16", ref_splits=1, tail_parts=1)
    for tp in (8, 0):
        got, st = run_knn(env, xq, xr, k, precision="fp16", ref_splits=1, tail_parts=tp)
        say("cross", tp, st)
        if tp:
            assert st["tail_parts"] == tp and 0 < st["tail_rows"] < len(xq)
            assert st["tile_launches"] == 2
        for u, v in zip(got, base):
            np.testing.assert_array_equal(u, v)
    oidx, odist = oracle.knn(xq, xr, k)
    compare_knn(xq, xr, np.arange(len(xq)), base[0], base[1], oidx, odist)


def test_query_blocks_each_split(env):
    """Query blocks: each block's tail is split on its own and the tail region
    is reused block after block."""
    _, _, oracle = env
    x, _ = workloads.generate("C2", n=11000)
    k = 20
    base, _ = run_knn(env, x, x, k, precision="fp16", exclude_self=True, ref_splits=1,
                      query_block=4096, tail_parts=1)
    got, st = run_knn(env, x, x, k, precision="fp16", exclude_self=True, ref_splits=1,
                      query_block=4096, tail_parts=6)
    say("blocks", st)
    assert st["blocks"] == 3 and st["tail_parts"] == 6 and st["tail_rows"] == len(x)
    for u, v in zip(got, base):
        np.testing.assert_array_equal(u, v)
    oidx, odist = oracle.knn_self(x, k)
    compare_knn(x, x, np.arange(len(x)), got[0], got[1], oidx, odist)


def test_short_scans_limit_pieces(env):
    """At least four stages per piece: 700 references (six stages of 128 rows
    at d = 32) allow one piece only, so no split happens."""
    rng = np.random.default_rng(8)
    x = rng.standard_normal((700, 32)).astype(np.float32)
    got, st = run_knn(env, x, x, 7, precision="fp16", exclude_self=True, ref_splits=1,
                      tail_parts=8)
    assert st["tail_parts"] == 1 and st["tail_rows"] == 0
    base, _ = run_knn(env, x, x, 7, precision="fp16", exclude_self=True, ref_splits=1,
                      tail_parts=1)
    for u, v in zip(got, base):
        np.testing.assert_array_equal(u, v)

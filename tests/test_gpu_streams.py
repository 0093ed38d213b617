"""Calls on different streams with different workspaces may overlap (the
library keeps no state between calls): two host threads, each on a stream of
its own, run the kNN and LOF entry points on different inputs at the same
time, and every result must equal the same call made alone."""
import sys
import threading

import numpy as np
import pytest

from paper_2110_14007_amd import workloads

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_two_threads_two_streams():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    from paper_2110_14007_amd import tod

    x1, _ = workloads.generate("C2", n=20000)
    x2, _ = workloads.generate("C1")
    a1 = torch.from_numpy(x1).cuda()
    a2 = torch.from_numpy(x2).cuda()
    torch.cuda.synchronize()
    say("serial reference runs")
    ref1 = [t.cpu().numpy() for t in tod.tod_knn(a1, a1, 20)]
    ref2 = [t.cpu().numpy() for t in tod.tod_lof(a2, 10)]
    torch.cuda.synchronize()

    results = {}
    errors = []

    def worker(name, fn):
        try:
            s = torch.cuda.Stream()  # default priority
            ws = tod.Workspace()
            out = []
            for _ in range(4):
                out.append([t.cpu().numpy() for t in fn(ws, s)])
            results[name] = out
        except Exception as e:  # reported below, after both threads end
            errors.append(repr(e))

    t1 = threading.Thread(target=worker, args=(
        "knn", lambda ws, s: tod.tod_knn(a1, a1, 20, workspace=ws, stream=s)))
    t2 = threading.Thread(target=worker, args=(
        "lof", lambda ws, s: tod.tod_lof(a2, 10, workspace=ws, stream=s)))
    say("two threads")
    t1.start()
    t2.start()
    t1.join()
    t2.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for got in results["knn"]:
        np.testing.assert_array_equal(got[0], ref1[0])
        np.testing.assert_array_equal(got[1], ref1[1])
    for got in results["lof"]:
        np.testing.assert_array_equal(got[0], ref2[0])
        np.testing.assert_array_equal(got[1], ref2[1])

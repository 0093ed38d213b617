"""MI355X (gfx950) kNN / LOF outlier-detection hot path of TOD (arXiv 2110.14007).

The compute lives in ``libtod.so`` (HIP kernels behind a C ABI, see
``include/tod.h``); :mod:`.tod` is its Python binding and :mod:`.workloads`
the seeded synthetic inputs.  ``tod_knn``, ``tod_knn_score``, ``tod_lof``,
``tod_plan`` and ``tod_workspace_size`` are re-exported lazily: touching them
imports the binding, which raises ImportError if the library is not built.
"""
_EXPORTS = ("tod_knn", "tod_knn_score", "tod_lof", "tod_plan", "tod_workspace_size", "options",
            "new_stats", "Workspace", "TodError")


def __getattr__(name):
    if name in _EXPORTS:
        from . import tod
        return getattr(tod, name)
    raise AttributeError(name)

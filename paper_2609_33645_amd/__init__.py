"""Pruned CTC head-and-loss hot path for MI355X (gfx950).

The computation lives in libprunedctc.so (HIP kernels behind the C ABI of
include/prunedctc.h); ``paper_2609_33645_amd.prunedctc`` is its Python binding.
``paper_2609_33645_amd.workloads`` draws seeded synthetic inputs.
"""

__all__ = ["prunedctc", "workloads", "pruned_ctc_fwd_bwd"]


def __getattr__(name):
    if name == "pruned_ctc_fwd_bwd":
        from .prunedctc import pruned_ctc_fwd_bwd
        return pruned_ctc_fwd_bwd
    if name in ("prunedctc", "workloads"):
        import importlib
        return importlib.import_module(f".{name}", __name__)
    raise AttributeError(name)

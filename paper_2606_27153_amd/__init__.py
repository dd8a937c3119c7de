"""MI355X-native single-GPU Muon optimizer step (DMuon, arXiv 2606.27153).

The step itself runs in the HIP library ``libmuon_mi355x.so`` built from
``csrc/``; this package is its thin Python binding (argument marshalling
only).  Importing the package does not load the library; the first use of
the binding does, and fails loudly if the library has not been built.
"""
__all__ = ["MuonPlan", "Muon", "load_library"]


def load_library():
    from . import _lib
    return _lib.load()


def __getattr__(name):
    if name in ("MuonPlan", "Muon"):
        from . import optim
        return getattr(optim, name)
    raise AttributeError(name)

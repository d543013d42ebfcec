"""MI355X (gfx950) implementation of MTGR's jagged dynamic-mask HSTU attention
with the gated Group-LayerNorm that follows it (arXiv 2505.18654, Sec. 4.2).

The computation lives in libmtgr_hstu.so (hand-written HIP kernels behind a C
ABI, see include/mtgr_hstu.h); `hstu` binds its entry points by name and `ops`
wraps them for torch device tensors.
"""
from . import hstu  # noqa: F401
from .hstu import MtgrError, MtgrLibraryMissing  # noqa: F401

__all__ = ["hstu", "ops", "MtgrError", "MtgrLibraryMissing"]


def __getattr__(name):
    if name == "ops":               # torch wrappers load lazily (torch is heavy to import)
        import importlib
        return importlib.import_module(".ops", __name__)
    raise AttributeError(name)

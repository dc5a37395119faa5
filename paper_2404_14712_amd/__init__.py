"""MI355X (gfx950) implementation of ORBIT's ViT hot path (arXiv 2404.14712).

The computation lives in the HIP library liborbit.so (C ABI: include/orbit.h);
this package only binds it (`_lib`), builds it (`build`) and sequences the
entry points of one forward+backward pass (`model`).
"""
from ._lib import EXPORTS, LIB_PATH, OrbitError, OrbitLib  # noqa: F401

_LIB = None


def load(path: str = LIB_PATH) -> OrbitLib:
    """Load the HIP library (raises if it has not been built)."""
    global _LIB
    if _LIB is None or _LIB.path != path:
        _LIB = OrbitLib(path)
    return _LIB

"""Batched what-if GPU-frequency selection (throttLL'eM, arXiv 2408.05235) on
AMD MI355X: projection, tree-ensemble prediction and selection as HIP kernels
behind the C ABI in include/tl.h.  ``api`` holds the Python binding."""
from .configs import CONFIGS, get_config  # noqa: F401

__all__ = ["CONFIGS", "get_config", "api", "synth"]


def __getattr__(name):
    if name in ("api", "synth", "build"):
        import importlib
        return importlib.import_module(f".{name}", __name__)
    raise AttributeError(name)

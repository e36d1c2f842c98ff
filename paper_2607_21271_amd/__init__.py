"""MI355X (gfx950) implementation of the Flash EQ-Linear layer (arXiv 2607.21271).

The compute lives in ``libeqlinear.so`` (hand-written HIP, C ABI in
``include/eqlinear.h``).  ``_lib`` is the ctypes binding with the ABI's own
names; ``ops`` wraps it for torch tensors (memory and streams only) and adds
an autograd Function and ``EQLinear`` module.  Submodules load lazily, and
using them without the built library raises.
"""

__all__ = ["_lib", "ops", "roofline"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module("." + name, __name__)
    raise AttributeError(name)

"""MI355X (gfx950) fused multi-sub-model LM head + cross-entropy + distillation.

The compute runs in ``libmls.so`` (HIP kernels behind a C ABI declared in
``include/mls.h``); this package only marshals arguments to it. Importing the
package does not load the library: :func:`distill` and the wrappers in
:mod:`.binding` load it on first use and raise if it is missing.
"""

__all__ = ["distill", "api", "binding", "workloads"]


def __getattr__(name):
    if name == "distill":
        from .api import distill
        return distill
    if name in ("api", "binding", "workloads"):
        import importlib
        return importlib.import_module(f".{name}", __name__)
    raise AttributeError(name)

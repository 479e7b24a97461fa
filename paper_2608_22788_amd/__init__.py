"""MI355X (gfx950) paged decode / speculative-verify attention.

The hot path is libtsattn.so (HIP kernels behind the C ABI in
include/ts_attn.h); ``binding`` is its ctypes wrapper.  ``synth`` is the
seeded input generator and imports nothing from the rest of the package.
The binding is loaded lazily so that ``synth`` can be used without a build.
"""

__all__ = ["binding", "device", "synth"]


def __getattr__(name):
    if name in ("binding", "device"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)

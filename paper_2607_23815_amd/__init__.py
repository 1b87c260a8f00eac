"""Paged prefix-reuse attention for MI355X (gfx950).

`lib` is the ctypes binding of libpkv.so (include/pkv.h); `path` holds the one-call helpers
that run the hot path (append -> prefill attention, append -> decode attention) on torch
device tensors. Importing `lib` fails loudly when the library has not been built."""
__all__ = ["lib", "path"]


def __getattr__(name):
    if name in ("lib", "path"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)

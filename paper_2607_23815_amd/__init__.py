"""Paged prefix-reuse attention for MI355X (gfx950).

`lib` is the ctypes binding of libpkv.so (include/pkv.h): argument marshalling only, every
step of the path runs in the library's HIP kernels. Importing `lib` fails loudly when the
library has not been built."""
__all__ = ["lib"]


def __getattr__(name):
    if name == "lib":
        import importlib
        return importlib.import_module(f"{__name__}.lib")
    raise AttributeError(name)

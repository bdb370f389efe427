"""gkv: MI355X-native graded KV-cache decode attention (Geodesia-KV hot path).

The compute lives in the HIP/C library ``_lib/libgkv.so`` (built by
``__graft_entry__.build()``); ``binding`` is a thin ctypes layer over its C ABI
that takes torch tensors for device memory and streams.  Importing this package
does not load the library; ``binding`` does, and raises if it is missing.
"""
__all__ = ["binding", "synth", "workloads"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)

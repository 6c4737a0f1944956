"""MI355X-native LampAttention forward pass (look-ahead mixed-precision FlashAttention).

`paper_2609_39361_amd.lamp` is the Python binding of the C-ABI library
`liblamp.so` (HIP kernels for gfx950).  The binding is imported lazily so that
the input generators in `paper_2609_39361_amd.workloads` can be used on a
machine without the library or a GPU.
"""

__all__ = ["lamp", "workloads"]


def __getattr__(name):
    if name in ("lamp", "workloads"):
        import importlib
        return importlib.import_module("." + name, __name__)
    raise AttributeError(name)

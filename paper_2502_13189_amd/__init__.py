"""MI355X-native MoBA causal prefill forward (Mixture of Block Attention,
arXiv 2502.13189).

The compute path is a HIP library (``libmoba.so``, C ABI in ``include/moba.h``);
this package is a thin ctypes binding around it.  Submodules load lazily so that
``paper_2502_13189_amd.inputs`` can be imported without the library.
"""
__all__ = ["forward", "dense_forward", "pool", "select", "route"]


def __getattr__(name):
    if name in __all__:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)

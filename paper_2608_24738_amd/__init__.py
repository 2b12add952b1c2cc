"""MI355X-native exact Euclidean distance transform (``distance_transform_edt``).

The compute path is the C-ABI library ``libtm_edt.so`` (hand-written HIP
kernels for gfx950, declared in ``include/tm_edt.h``); ``binding`` marshals
torch tensors into it.  Importing the package loads nothing: the library is
opened on first use and a missing library is an error, never a fallback.
"""
__all__ = ["tm_edt", "tm_edt_sq", "tm_strerror", "distance_transform_edt",
           "distance_transform_edt_sq", "TMError"]


def __getattr__(name):
    if name in __all__:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)

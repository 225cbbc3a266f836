"""MI355X (gfx950) FastEagle cascaded drafter: HIP kernels behind a C ABI
(include/fe.h, libfe.so) and a thin ctypes binding.

    from paper_2509_20416_amd import fe          # C-ABI binding, same names as fe.h
    from paper_2509_20416_amd import Drafter     # torch device-memory plumbing
"""
from . import fe  # noqa: F401


def __getattr__(name):
    if name in ("Drafter", "DeviceInputs", "to_device"):
        from . import drafter
        return getattr(drafter, name)
    raise AttributeError(name)

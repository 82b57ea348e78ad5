"""MI355X (gfx950) routed mixture-of-head attention (NAMOH) hot path.

``route``, ``attn_fwd`` and ``decode_step`` call the C ABI of the in-tree
HIP library ``libnamoh.so`` (see include/namoh.h); ``workloads`` holds the
seeded synthetic input generators.  Importing the package does not load the
library or torch; the first call of a binding does.
"""


def __getattr__(name):
    if name in ("route", "attn_fwd", "decode_step", "lib", "NamohError"):
        from . import _lib
        return getattr(_lib, name)
    raise AttributeError(name)

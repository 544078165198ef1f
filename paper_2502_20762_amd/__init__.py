"""ncodec: MI355X (gfx950) HIP implementation of the DCVC-RT per-frame transform.

The product is ``libncodec.so`` (C ABI in ``include/ncodec.h``); this package
holds its HIP sources (``csrc/``), the in-tree build (``build.py``) and the
ctypes binding (``ncodec.py``).
"""
from .ncodec import (Codec, NcodecError, load_library, make_config,  # noqa: F401
                     ncodec_config)

"""MI355X (gfx950) streaming KV step of acoustic-to-text KV compression.

The work runs in libA2T (HIP kernels behind the C ABI of include/a2t.h);
this package is its ctypes binding, with the same call names.  Importing it
without a built libA2T.so raises ImportError: build it with
``python paper_2609_31224_amd/build.py``.
"""
from ._lib import *  # noqa: F401,F403
from ._lib import (A2TError, Cache, EXPORTED, LIB_PATH, a2t_config,  # noqa: F401
                   a2t_stream_info)

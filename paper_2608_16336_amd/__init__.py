"""Multi-tier Llumnix scheduling step on MI355X.

The compute path is the HIP library ``_lib/libmts.so`` (C ABI declared in
``include/mts.h``); :mod:`paper_2608_16336_amd.mts` is a thin ctypes binding
with the same function names.  There is no CPU fallback: using the binding
without the built library raises.
"""
from .mts import (MtsError, Scheduler, load_library, make_cfg,  # noqa: F401
                  mts_state_bytes, NSTAT)

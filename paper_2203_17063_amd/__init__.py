"""libecc on MI355X: eventually consistent (stale-synchronous) collectives on
P virtual ranks in one GPU's HBM, and the block-row iterations they feed.

The compute path is the HIP library ``libecc.so`` (sources in ``csrc/``,
interface in ``include/libecc.h``); ``capi`` is its ctypes binding and
``runner`` uploads arrays with torch and drives the C ABI.
"""
from . import capi  # noqa: F401

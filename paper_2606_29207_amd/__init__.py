"""MI355X (gfx950) hot path of KernelFlume's weightless attention node.

``kf``   -- ctypes binding of libkf.so (include/kf.h): tail append, partial
            attention over token-range routes, log-sum-exp merge.
``step`` -- device-resident decode state that runs the three calls in order.
``build``-- hipcc build of libkf.so.
"""
from . import kf  # noqa: F401

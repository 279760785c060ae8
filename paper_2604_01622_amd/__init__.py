"""MI355X-native expert-choice (EC) mixture-of-experts layer.

The computation lives in libecmoe.so (HIP for gfx950, C interface in
include/ec_moe.h).  This package is its thin Python binding: argument
marshalling with torch tensors as device buffers and torch's current stream.
Every step of the layer runs in the library's kernels; there is no fallback.
"""
from .binding import (  # noqa: F401
    ECError,
    Problem,
    backward,
    capacity,
    forward,
    lib,
    route,
    route_noalloc,
    saved_views,
    token_coverage,
    tc_capacity,
    tc_route,
    tc_forward,
    Layer,
    TcLayer,
)

__all__ = ["ECError", "Problem", "Layer", "TcLayer", "route", "route_noalloc", "forward", "backward", "capacity",
           "saved_views", "token_coverage", "tc_capacity", "tc_route", "tc_forward", "lib"]

"""CPU float64 oracle of the expert-choice MoE layer (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg import this
package; the HIP library and its Python binding never do.
"""
from .ec_ref import *  # noqa: F401,F403

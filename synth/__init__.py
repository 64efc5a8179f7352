"""Seeded synthetic inputs for the AEP expert-layer path.

This package only draws random numbers and stores them in the element formats
the path consumes (f32, bf16 bit patterns, OCP e4m3fn codes plus per-channel
scales).  It holds none of the MoE layer's arithmetic (no routing, queueing,
FFN or combine), so the CPU oracle and the HIP path can both take their inputs
from it without sharing any of the method.
"""

from .workloads import *  # noqa: F401,F403
from .arrivals import *  # noqa: F401,F403

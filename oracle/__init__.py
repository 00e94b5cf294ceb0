"""CPU float64 oracle of the renderer-attention path (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package.  It shares no code with the HIP library or its binding.
"""
from .ff_oracle import *  # noqa: F401,F403

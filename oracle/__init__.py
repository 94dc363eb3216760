"""CPU oracle for the ACID-gated video-DiT denoise loop (test infrastructure).

This package is test infrastructure: only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it.  It shares no code with the HIP
library and never imports it.
"""
from .acid_oracle import *  # noqa: F401,F403

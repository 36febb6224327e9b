"""Float64 CPU oracle for the sparse sequence-parallel attention hot path.

TEST INFRASTRUCTURE ONLY. Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this package. The product path (the
HIP library and its Python binding) never calls into it and shares no code
with it.
"""

from .sparsp_oracle import *  # noqa: F401,F403
from .sparsp_oracle import __all__  # noqa: F401

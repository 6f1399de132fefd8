"""CPU oracle for the BinaryPC decode hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import anything from this package.  The product path (the HIP library and its
Python binding) never calls into it, and it never calls into the product
path: the two share no code, headers, tables or helpers.
"""

from .bpc_oracle import *  # noqa: F401,F403
from .bpc_oracle import __all__  # noqa: F401

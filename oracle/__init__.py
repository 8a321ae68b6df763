"""fp64 CPU oracle for the product-key memory hot path (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg use this
package.  The product path never imports it.
"""
from .pkm_oracle import *  # noqa: F401,F403
from .pkm_oracle import __all__  # noqa: F401

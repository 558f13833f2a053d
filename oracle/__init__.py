"""Float64 CPU oracle of the Hierarchical Global Attention routed-attention path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything in this package; only
the test suite, the smoke check and the CPU-baseline leg of the benchmark use
it.  It shares no code with the HIP path.
"""

from .hga_oracle import *  # noqa: F401,F403

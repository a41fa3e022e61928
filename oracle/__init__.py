"""fp64 CPU oracle for Nystrom-approximated Laplacian-kernel attention.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this package.  The product path (the HIP
library and its binding) never loads it, and the two share no code.

The arithmetic lives in ``lapattn_oracle.c`` (plain fp64 loops); this module only
builds it with gcc and marshals numpy arrays through ctypes.
"""
from .oracle import (  # noqa: F401
    build,
    load,
    kernel,
    segments,
    windows,
    ns,
    forward,
    backward,
    dwc,
    dwc_backward,
    threads,
    NORM_INLINE,
    NORM_ROWSUM,
    NORM_NONE,
    NORM_MSPACE,
)

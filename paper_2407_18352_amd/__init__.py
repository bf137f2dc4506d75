"""MI355X-native surrogate-inference region of HPAC-ML (arXiv 2407.18352).

The product is ``libhpacml.so`` (C ABI in ``include/hpacml.h``, HIP kernels for
gfx950).  ``api`` is a thin ctypes binding over it; ``workloads`` draws the
seeded synthetic inputs.  Nothing here falls back to a CPU path: without the
built library every call raises.
"""
from ._abi import (ACT_IDENTITY, ACT_RELU, BF16, BND_CLAMP, BND_NONE, BND_PERIODIC, F32, FROM, TO,
                   HpacmlError)

__all__ = ["ACT_IDENTITY", "ACT_RELU", "BF16", "BND_CLAMP", "BND_NONE", "BND_PERIODIC", "F32", "FROM",
           "TO", "HpacmlError"]

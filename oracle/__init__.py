"""CPU oracle for the region-reuse DiT step (RegionCache).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  The product path never calls it,
and it shares no code with the HIP library.

The oracle is plain NumPy, float64 by default, written from the paper:
edit-region localisation from cross-attention (Sec. 3.2), the hidden-state
cache pool (Sec. 3.2), region-level sparse attention with the merge of active
outputs into cached inactive states (Sec. 3.3), the reuse cutoff (Sec. 3.3,
Eq. 1 and Eq. 2) and the fused K/V scatter that writes fresh active keys and
values into the cached positions before attention reads them (Sec. 3.4,
"Kernel Fusing").  The model internals follow the public PixArt-alpha block
the paper evaluates (Sec. 4.1).
"""
from .rc_oracle import *  # noqa: F401,F403
from .rc_oracle import __all__  # noqa: F401

"""Float64 CPU oracle of the low-rank compressor with error feedback.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the GPU library (no kernels, headers, helpers or constants).
"""

from .powerlr import (RANK_TOL, compress, decompress, err_update, lift, mgs2,
                      step, step_batched)

__all__ = ["RANK_TOL", "compress", "decompress", "err_update", "lift", "mgs2",
           "step", "step_batched"]

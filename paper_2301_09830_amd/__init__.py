"""liboptcc: MI355X-native low-rank power-iteration compressor with error feedback.

The compute path is the HIP library liboptcc.so (csrc/); `optcc` is its thin
ctypes binding over torch tensors.  Build the library with
`python -m paper_2301_09830_amd.build`.
"""

from . import optcc  # noqa: F401
from .optcc import (OCC_BF16, OCC_DEC_OUT_BF16, OCC_DEC_SPLIT_BF16, OCC_F32,  # noqa: F401
                    OCC_F_BAD_ROWS, OCC_F_NONFINITE, OCC_F_RANK_DEFICIENT, OCC_NO_MHAT, OccError,
                    alloc_workspace, occ_abi_version, occ_compress,
                    occ_compress_workspace_bytes, occ_decompress, occ_decompress_ex,
                    occ_err_update, occ_get_flags, occ_pipeline_1f1b, occ_profile_begin,
                    occ_profile_end, occ_sc_select, occ_status_str, occ_step, occ_step_batched,
                    occ_step_batched_noalloc, occ_step_rows, occ_step_rows_workspace_bytes,
                    occ_workspace_bytes, occ_workspace_init)

"""MI355X (gfx950) read-sparse memory readout and store-sparse commit.

Python binding of the rs3 C ABI (include/rs3.h).  Every step of the path runs
in the HIP kernels of librs3.so; this package only marshals arguments.  It
fails loudly when the library is missing: there is no fallback.
"""
from ._binding import (  # noqa: F401
    RS3_OK, RS3_E_INVALID, RS3_E_CAPACITY, RS3_E_DEVICE, RS3_E_OOM,
    RS3_F32, RS3_BF16, RS3_MAX_OBJ, RS3_MAX_MN, RS3_TRACK_WORDS, RS3_BANK_HDR_WORDS, RS3_NOALLOC_SCRATCH_BYTES,
    Rs3Error, lib, lib_path, exported_symbols, Grid, SelectParams, FrameIO,
    Track, Layer, Bank, Stack, StackWeights,
    select_workspace_size, select_queries,
    readout_workspace_size, readout, readout_noalloc, commit, frame_workspace_size, frame, readout_commit, write_keepset, close_workspace_size, close_masks,
    attend_workspace_size, attend,
    KERNEL_NAMES, profile_enable, profile_reset, profile_report, RS3_STREAM_READ_THREADS, stream_read,
)

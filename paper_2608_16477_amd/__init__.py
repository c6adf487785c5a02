"""MI355X (gfx950) library for target-side KV-cache reconstruction.

The compute lives in ``libpallas.so`` (hand-written HIP kernels behind a C
ABI declared in ``include/pallas.h``); this package is the thin ctypes
binding that marshals torch device tensors into those calls.  Importing the
binding does not touch the GPU; the first call loads the library and fails
loudly if it has not been built.
"""
from .binding import (  # noqa: F401
    PallasError, Status, lib, library_path,
    pallas_abi_version, pallas_last_error, pallas_check_coverage,
    pallas_model_create, pallas_model_destroy, pallas_workspace_size,
    pallas_prefill_prefix, pallas_prefill_chunk, pallas_pack_suffix_blocks, pallas_assemble_kv,
    pallas_decode_step, pallas_decode_step_static, Model, ChunkDesc, ChunkHeader, EXPORTS, KERNEL_CLASSES,
    pallas_profile_enable, pallas_profile_read, pallas_profile_reset, pallas_profile_clock,
    pallas_window_select, pallas_window_evaluate, pallas_ewma_update, pallas_admit,
    pallas_waste_bound, WindowParams, WindowDecision, Ewma,
)

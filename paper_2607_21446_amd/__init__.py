"""MI355X (gfx950) KroQuant online activation quantizer.

The compute lives in libkroquant.so (hand-written HIP, C ABI in
include/kroquant.h); this package is its thin Python binding.
"""
from .binding import (  # noqa: F401
    CALIB_NOALLOC_MAX_BYTES, EXPORTED, PACK_BYTES_PER_FACTOR, KQError, calib_reference, calib_step,
    calib_step_noalloc, calib_workspace, calibrate, e2m1_encode, factors_inverse_transpose, fwht, hadamard32, hadamard_lu, lib, lu_to_factors, mxfp4, mxfp4_gemm,
    pack_factors, quantize, quantize_exact, quantize_lu, quantize_packed, smoothquant, status_string, stream_floor,
    stream_probe, TIMESTAMP_HZ, timestamp,
    version,
    weight_transform,
)

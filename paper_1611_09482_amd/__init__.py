"""Fast Wavenet cached generation on AMD MI355X (gfx950).

The compute path is the C-ABI library libfwg.so (HIP kernels); this package is
a thin ctypes binding with the same names.  PyTorch supplies device memory and
streams only.
"""
from .binding import (FWG_BF16, FWG_F32, FWG_GATED, FWG_RELU, FWG_RELU_RESIDUAL, FastWavenet, FwgError, from_model,
                      load_library, upload_weights)

__all__ = ["FastWavenet", "FwgError", "load_library", "from_model", "upload_weights", "FWG_RELU", "FWG_RELU_RESIDUAL", "FWG_GATED",
           "FWG_F32", "FWG_BF16"]

"""MI355X (gfx950) implementation of the H-Scale hot path.

H-Scale refines NVFP4 per-group scales with a diagonal second-order proxy:
``hdiag`` computes h = diag(X^T X) from calibration activations and
``search`` picks, for every 16-weight group, the E4M3 scale among a window of
neighbours of the max-abs scale that minimises the h-weighted reconstruction
error, returning NVFP4 scale bytes and packed E2M1 codes.

The compute is in ``libhscale.so`` (hand-written HIP, C ABI in
``include/hscale.h``); this package is its thin Python binding.
"""
from ._lib import HScaleError, EXPORTS  # noqa: F401
from .ops import (hdiag, hdiag_accumulate, hdiag_finalize, hdiag_noalloc, hdiag_workspace_bytes, quantize,  # noqa: F401
                  output_error, output_error_workspace_bytes, search, search_block, search_layers, search_stats,
                  shift_summary)

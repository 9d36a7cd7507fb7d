"""CoSpec verify-and-arbitrate step on MI355X (gfx950).

The computation runs in libcospec.so (HIP kernels behind the C ABI of
include/cospec.h); `binding` marshals torch tensors into it, `workloads` draws
seeded synthetic inputs.
"""
from .binding import (CospecError, SplitBlock, arbitrate, hybrid_attention, hybrid_mask, lib,
                      prepare_block, prepare_sps, prepare_tree, sps_block, verify_block, verify_block_static,
                      verify_tree)

__all__ = ["CospecError", "SplitBlock", "arbitrate", "hybrid_attention", "hybrid_mask", "lib",
           "prepare_block", "prepare_sps", "prepare_tree", "sps_block", "verify_block", "verify_block_static",
           "verify_tree"]

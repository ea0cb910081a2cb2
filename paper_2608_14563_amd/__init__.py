"""MI355X-native FPO hot path: output-projected pseudogradient and update.

The compute path is the HIP library `libfpo.so` (C ABI declared in
include/fpo.h); `paper_2608_14563_amd.api` marshals torch tensors into it.
Importing this package does not load the library; the first API call does,
and fails loudly if it is missing.
"""
__all__ = ["api", "inputs"]

"""MI355X-native IKBO inference hot path of ROCS (arXiv 2607.27744).

The computation lives in librocs.so (hand-written HIP kernels for gfx950 behind
the C ABI declared in include/rocs.h). This package only marshals torch device
tensors into that ABI (`ops`), loads the library (`_lib`), builds it (`build`)
and draws seeded synthetic inputs (`workloads`). Importing the package does not
load the library; the first operator call does, and fails loudly if it is
missing.
"""

__all__ = ["ops", "workloads"]

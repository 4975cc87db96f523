"""RNN-Transducer and W-Transducer loss + gradient on the T x (U+1) grid lattice,
for AMD Instinct MI355X (gfx950).

The work is done by HIP kernels in librnnt_mi355x.so behind the C-ABI in
include/rnnt_mi355x.h (the loss and its gradient, forced alignment on the same
lattices, and the loss over any lattice given as an arc list); this package is
the thin Python binding.
"""
from .binding import (ArcPlan, RNNTError, arc_loss, arc_loss_workspace_bytes, arc_plan, lattice_scores,  # noqa: F401
                      load_library, log_softmax_gather, loss_workspace_bytes, rnnt_loss, rnnt_loss_noalloc, status_string,
                      version, viterbi_align, viterbi_workspace_bytes)
from . import topologies  # noqa: F401
from .autograd import RNNTLoss, rnnt_loss_autograd  # noqa: F401

__all__ = ["rnnt_loss", "rnnt_loss_noalloc", "log_softmax_gather", "lattice_scores", "loss_workspace_bytes", "RNNTLoss",
           "rnnt_loss_autograd", "RNNTError", "load_library", "status_string", "version", "viterbi_align",
           "viterbi_workspace_bytes", "arc_plan", "arc_loss", "arc_loss_workspace_bytes", "ArcPlan", "topologies"]

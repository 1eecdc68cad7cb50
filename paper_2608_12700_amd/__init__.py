"""MI355X-native (gfx950) gated-delta-rule chunked forward and training backward.

The work runs in hand-written HIP kernels behind the C ABI of include/gdn.h
(libgdn.so, built in-tree by ``python -m paper_2608_12700_amd.build``).
``paper_2608_12700_amd.gdn`` is the thin Python binding;
``paper_2608_12700_amd.autograd.gated_delta_rule`` wraps it for torch autograd.
"""
from .gdn import (EXPORTED, GdnError, Packed, bwd, fwd, gdn_bwd, gdn_bwd_workspace_size, gdn_fwd,
                  gdn_fwd_workspace_size, gdn_num_chunks, gdn_status_str, gdn_version, load,
                  make_problem)

__all__ = ["fwd", "bwd", "gdn_fwd", "gdn_bwd", "gdn_num_chunks", "gdn_fwd_workspace_size",
           "gdn_bwd_workspace_size", "gdn_status_str", "gdn_version", "load", "make_problem",
           "Packed", "GdnError", "EXPORTED"]

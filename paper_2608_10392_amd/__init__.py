"""MI355X (gfx950) implementation of the forward pass of one UniF-MoE
feed-forward layer ("Share First, Route What Remains", Sec. III).

The computation lives in the HIP library libunifmoe.so (C ABI in
include/unif_moe.h); this package is its thin Python binding. The library is
loaded on first use and its absence is an error.
"""
from ._lib import (  # noqa: F401
    UnifMoeError, alloc_routing, alloc_workspace, block_forward, block_forward_workspace_size,
    layer_backward, layer_backward_workspace_size, layer_forward,
    layer_forward_workspace_size, lib, make_config, route, route_workspace_size, stats,
    stats_workspace_size, status_string,
)

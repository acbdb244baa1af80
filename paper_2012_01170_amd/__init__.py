"""sbconv: sparse basis convolution on continuous domains for MI355X (gfx950).

The compute path is the HIP library libsbconv.so behind the C ABI declared in
include/sbconv.h; this package is its thin torch binding.
"""
from .ops import (CSC, CSR, Geometry, basis_eval, conv_backward, conv_forward,
                  conv_forward_noalloc, conv_forward_noalloc_max_bytes, conv_plan, conv_workspace_size, csr_transpose, csr_transpose_batched,
                  conv_decay_gradient, featureless_backward, featureless_forward, sample_points,
                  lif_sample_events, EventStream,
                  neighbour_search_events, neighbour_search_events_csc,
                  neighbour_search_points, resolve_order)

__all__ = ["CSC", "CSR", "Geometry", "basis_eval", "conv_backward", "conv_forward",
           "conv_forward_noalloc", "conv_forward_noalloc_max_bytes", "conv_plan", "conv_workspace_size", "csr_transpose", "csr_transpose_batched",
           "conv_decay_gradient", "featureless_backward", "featureless_forward", "sample_points",
           "lif_sample_events", "EventStream",
           "neighbour_search_events", "neighbour_search_events_csc",
           "neighbour_search_points", "resolve_order"]

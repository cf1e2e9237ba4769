"""Masked co-adaptive MoE layer (MaskCoFT) on AMD Instinct MI355X.

The hot path lives in ``libmaskmoe.so`` (hand-written HIP for gfx950, C ABI in
``include/maskmoe.h``); ``_lib`` is its ctypes binding and ``synth`` the seeded
input generator. Importing the package does not load the library; the first
call into ``_lib`` does, and fails loudly if it has not been built.
"""

from ._lib import (BF16, CACHE_FIFO, CACHE_LFU, CACHE_LRU, F32, GATE_P, GATE_RENORM, LAYOUT_PACKED,  # noqa: F401
                   LAYOUT_ROWS, ROUTE_HARD_MASK, ROUTE_PLAIN,
                   ROUTE_SOFT_PRIOR, LayerDesc, MaskMoEError, load, make_desc, maskmoe_cache_fetches,
                   maskmoe_layer_forward, maskmoe_layer_workspace_bytes, maskmoe_pack_expert_weights, maskmoe_route)

"""MI355X (gfx950) implementation of the MoEBlaze MoE layer hot path
(arXiv 2601.05296): routing, buffer-free dispatch, gather-fused grouped SwiGLU
GEMMs with SiLU recomputation, and the gate-weighted combine, forward and
backward, behind the C ABI in include/moeblaze.h.

`binding` exposes the C entry points one-to-one; `layer` chains them into one
layer's forward and backward; `synth` draws the seeded synthetic inputs.
"""
from .binding import (EXPORTS, MOE_ACCUMULATE, MOE_BF16, MOE_F32, MOE_RENORM, MoEError,  # noqa: F401
                      load_library, moe_build_index, moe_build_index_workspace_size,
                      moe_combine, moe_ffn_bwd, moe_ffn_bwd_workspace_size, moe_ffn_fwd,
                      moe_ffn_fwd_workspace_size,
                      moe_route, moe_route_bwd, moe_route_bwd_workspace_size)

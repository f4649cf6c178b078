"""MI355X-native triangle self-attention (MegaFold's memory-efficient 3D
attention, arXiv 2506.20686): a C-ABI library over gfx950 HIP kernels
(libtriattn.so) and this thin Python binding."""
from .binding import (BF16, ENDING, F32, STARTING, TriAttnError, TriangleAttention, bwd, fwd,
                      tri_attn_bwd, tri_attn_bwd_workspace_bytes, tri_attn_fwd,
                      tri_attn_fwd_workspace_bytes, tri_attn_status_string, triangle_attention)

__all__ = ["BF16", "ENDING", "F32", "STARTING", "TriAttnError", "TriangleAttention", "bwd",
           "fwd", "tri_attn_bwd", "tri_attn_bwd_workspace_bytes", "tri_attn_fwd",
           "tri_attn_fwd_workspace_bytes", "tri_attn_status_string", "triangle_attention"]

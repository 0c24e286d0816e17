"""Hidden Decoding hot path on AMD MI355X: stream expansion and Stream-Factorized
Attention (forward and backward) as hand-written HIP kernels for gfx950, exposed
through the C ABI of include/hd.h (libhd.so) and this thin Python binding.

The library is loaded lazily on the first call; a missing build raises ImportError.
"""
from .binding import (HD_DTYPE_BF16, HD_DTYPE_F32, HD_SFA_INTRA, HD_SFA_LOCAL,
                      HD_SFA_MIX, HDError, cyclic_replicate, expand_embed,
                      expand_embed_backward, final_stream_gather, final_stream_gather_backward, hd_cyclic_replicate,
                      hd_embed_grad_scatter_add, hd_expand_embed, hd_expand_embed_bwd, hd_expand_embed_bwd_workspace_bytes,
                      hd_final_stream_gather, hd_final_stream_gather_bwd, hd_sfa_bwd, hd_sfa_bwd_final,
                      hd_sfa_bwd_final_workspace_bytes, hd_sfa_bwd_local, hd_sfa_bwd_local_workspace_bytes, hd_sfa_bwd_workspace_bytes,
                      hd_sfa_bwd_min_workspace_bytes, hd_sfa_bwd_local_min_workspace_bytes,
                      hd_sfa_bwd_final_min_workspace_bytes,
                      hd_sfa_decode, hd_sfa_decode_noalloc, hd_sfa_decode_noalloc_max_bytes,
                      hd_sfa_decode_workspace_bytes, hd_sfa_fwd, hd_sfa_fwd_final,
                      hd_sfa_fwd_local, hd_timing_collect, hd_timing_enable, hd_timing_filter,
                      sfa_backward, sfa_decode, sfa_final_backward, sfa_final_forward,
                      sfa_forward)

__all__ = ["HD_DTYPE_BF16", "HD_DTYPE_F32", "HD_SFA_INTRA", "HD_SFA_LOCAL",
           "HD_SFA_MIX", "HDError", "cyclic_replicate", "expand_embed",
           "expand_embed_backward", "final_stream_gather", "final_stream_gather_backward", "hd_cyclic_replicate",
           "hd_embed_grad_scatter_add", "hd_expand_embed", "hd_expand_embed_bwd", "hd_expand_embed_bwd_workspace_bytes",
           "hd_final_stream_gather", "hd_final_stream_gather_bwd", "hd_sfa_bwd", "hd_sfa_bwd_final",
           "hd_sfa_bwd_final_workspace_bytes", "hd_sfa_bwd_local", "hd_sfa_bwd_local_workspace_bytes", "hd_sfa_bwd_workspace_bytes",
           "hd_sfa_bwd_min_workspace_bytes", "hd_sfa_bwd_local_min_workspace_bytes",
           "hd_sfa_bwd_final_min_workspace_bytes",
           "hd_sfa_decode", "hd_sfa_decode_noalloc", "hd_sfa_decode_noalloc_max_bytes",
           "hd_sfa_decode_workspace_bytes", "hd_sfa_fwd", "hd_sfa_fwd_final",
           "hd_sfa_fwd_local", "hd_timing_collect", "hd_timing_enable", "hd_timing_filter",
           "sfa_backward", "sfa_decode", "sfa_final_backward", "sfa_final_forward",
           "sfa_forward"]


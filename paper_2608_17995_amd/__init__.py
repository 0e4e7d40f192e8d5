"""AViTS selective-upsampling step on MI355X: Python binding of libavits.so.

Argument marshalling only.  Every entry point mirrors the C function of the
same name in include/avits.h: tensors are passed as device pointers, the
stream is torch's current HIP stream, and a non-zero return code raises
AvitsError.  Every computation runs in the HIP kernels of libavits.so; there
is no CPU fallback, and calling any entry point without the built library
raises.
"""
from ._binding import (  # noqa: F401
    AvitsError, load, lib_path, version,
    F32, BF16, UP_NEAREST, UP_BILINEAR, BLOCK_DOUBLE, BLOCK_SINGLE,
    avits_score_workspace_bytes, avits_score, avits_score_select, avits_score_batched_workspace_bytes,
    avits_score_batched,
    avits_select_workspace_bytes, avits_select, avits_select_perturbed, avits_select_batched,
    avits_select_noalloc, avits_select_noalloc_max_n,
    avits_gather_upsample, avits_gather_upsample_ln, avits_scatter, avits_joint_lse, avits_gather_upsample_batched,
    avits_scatter_batched,
    avits_block_workspace_bytes, avits_block_forward, avits_block_forward_ex, avits_block_forward_batched,
    avits_block_forward_batched_ex,
    BlockWeights,
    avits_block_qk_workspace_bytes, avits_block_qk,
    avits_joint_attention_stats, avits_score_from_mass,
    avits_gather_mixed, avits_scatter_mixed,
    avits_linear, avits_final_layer_workspace_bytes, avits_final_layer, avits_euler_update,
    avits_noise_reinject, avits_noise_bits, NOISE_RASTER, NOISE_HALF_UNITS, NOISE_LOWRES,
    avits_grid_positions, avits_scale_positions,
    avits_timing_enable, avits_timing_reset, avits_timing_read,
)

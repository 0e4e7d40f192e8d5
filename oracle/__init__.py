"""CPU oracle for the AViTS selective-upsampling step.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 NumPy
statement of what the hot path computes, written from the paper (Section 3.3,
Eqs. spatial / dit_attn / zbar / step_var / joint / topk, and the joint
image-text attention block of Section 3.3.1).  Only the tests, the smoke check
and the benchmark's CPU-baseline leg import it.  The product path (the HIP
library and its Python binding) never imports, calls or links anything here,
and this package imports nothing from the product path.

Readings of the paper taken where it is silent or ambiguous are stated in the
docstrings of the functions they affect.  Every function here is pinned by the
CPU tests against brute force, closed forms, library special cases or
invariants; none is marked unpinned.
"""
from .importance import (  # noqa: F401
    spatial_importance, spatial_importance_bruteforce, joint_lse, step_variance,
    minmax_normalise, joint_score, score, text_attention_mass, score_from_mass,
)
from .selection import select_topk, select_topk_perturbed, select_topk_batched  # noqa: F401
from .relayout import (  # noqa: F401
    upsample_nearest, upsample_bilinear, gather_upsample, scatter, selected_positions,
    mixed_layout, gather_mixed, scatter_mixed,
)
from .block import (  # noqa: F401
    layer_norm, rms_norm, rope_angles, apply_rope, attention, gelu_tanh,
    double_block, single_block, block_qk, block_batched,
)
from .sampler import linear, final_layer, euler_update, euler_integrate  # noqa: F401
from .noise import (  # noqa: F401
    philox4x32_10, box_muller, pixel_noise_bits, pixel_noise, block_noise, halfunit_noise, reinject,
)

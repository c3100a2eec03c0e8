"""CPU oracle for the BEVPoolv2 view-transform path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 numpy code written from the paper's definition of the
Lift-Splat-Shoot view transformation (BEVPoolv2, section 2.1): materialise the
(N, D, H, W, C) frustum feature from the depth score and the image feature,
drop frustum points outside every voxel, and sum the remaining points into
the voxel their index names.  It shares no code with the HIP path and must
only be imported by the tests, by the smoke check and by the benchmark's CPU
baseline leg; the product path never calls it.
"""

from .bevpool_ref import (
    kept_mask,
    point_ranks,
    prepare_ref,
    frustum_feature,
    forward_ref,
    backward_ref,
    forward_cells_ref,
    grad_depth_points_ref,
    grad_feat_pixels_ref,
    depth_lse_ref,
    depth_softmax_ref,
    forward_softmax_ref,
    geometry_ref,
)

__all__ = [
    "kept_mask",
    "point_ranks",
    "prepare_ref",
    "frustum_feature",
    "forward_ref",
    "backward_ref",
    "forward_cells_ref",
    "grad_depth_points_ref",
    "grad_feat_pixels_ref",
    "depth_lse_ref",
    "depth_softmax_ref",
    "forward_softmax_ref",
    "geometry_ref",
]

"""Seeded synthetic inputs for the BEVPoolv2 view-transform path.

This package produces the *inputs* of the method and nothing else: the
camera-rig voxel index of every frustum point (``coor``), the depth score,
the image feature and an upstream gradient.  It holds none of the method's
own arithmetic (no filtering, rank formation, sorting, interval detection,
pooling or gradients), so both the CPU oracle and the HIP path can consume
the same inputs without sharing any code that computes a result.

Shapes follow BEVPoolv2 section 2.1: depth score (N, D, H, W), image feature
(N, H, W, C), with a leading batch axis B added here.
"""

from .configs import CONFIGS, Config, get_config
from .rig import frustum_coor, frustum_params, jittered_cameras, random_coor, rig_cameras
from .data import draw_inputs, draw_small

__all__ = [
    "CONFIGS",
    "Config",
    "get_config",
    "frustum_coor",
    "random_coor",
    "rig_cameras",
    "jittered_cameras",
    "frustum_params",
    "draw_inputs",
    "draw_small",
]

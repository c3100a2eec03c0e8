"""Voxel index of every frustum point for the synthetic camera rig.

BEVPoolv2 section 2.1 takes the voxel index of each frustum point as a given
input, computed offline from the camera intrinsics and extrinsics; the method
itself starts from that index.  This module plays the role of that offline
producer for an idealised rig, in float64:

* intrinsics: focal f = (W_img/2) / tan(hFOV/2), square pixels, principal
  point at the image centre (cx, cy) = (W_img/2, H_img/2);
* feature cell (h, w) sits at the pixel centre u = (w+0.5)*stride,
  v = (h+0.5)*stride;
* depth bin k is at depth_start + k*depth_step, measured along the optical
  axis;
* camera frame (x right, y down, z forward) to ego frame (x forward, y left,
  z up): x0 = Zc, y0 = -Xc, z = -Yc + cam_height, then a yaw of n*60 deg
  about the ego z axis;
* voxel index = floor((coordinate - lower bound) / cell size), half-open
  range; points outside the grid keep their out-of-range index so that the
  method's own filtering step decides what to drop.

The result is ``coor``: int32 (P, 3) holding (x, y, z) voxel indices, with
points enumerated p = (((b*N + n)*D + d)*H + h)*W + w, the same layout as the
depth score.  All B samples share the rig.
"""

from __future__ import annotations

import math

import numpy as np

from .configs import Config


def _floor_index(values: np.ndarray, lo: float, res: float) -> np.ndarray:
    idx = np.floor((values - lo) / res)
    # Keep far-away points representable; anything this large is out of range
    # for every grid used here and is filtered by the method.
    idx = np.clip(idx, -(2 ** 30), 2 ** 30)
    return idx.astype(np.int64)


def frustum_coor(cfg: Config) -> np.ndarray:
    """int32 (B*N*D*H*W, 3) voxel index (x, y, z) of every frustum point."""
    N, D, H, W = cfg.N, cfg.D, cfg.H, cfg.W
    f = cfg.focal
    cx = cfg.img_w / 2.0
    cy = cfg.img_h / 2.0
    u = (np.arange(W, dtype=np.float64) + 0.5) * cfg.stride          # (W,)
    v = (np.arange(H, dtype=np.float64) + 0.5) * cfg.stride          # (H,)
    dep = cfg.depth_start + np.arange(D, dtype=np.float64) * cfg.depth_step  # (D,)

    d3 = dep[:, None, None]
    Xc = ((u[None, None, :] - cx) * d3) / f       # (D, 1, W)
    Yc = ((v[None, :, None] - cy) * d3) / f       # (D, H, 1)
    Zc = d3                                       # (D, 1, 1)
    x0 = np.broadcast_to(Zc, (D, H, W))
    y0 = np.broadcast_to(-Xc, (D, H, W))
    z = np.broadcast_to(-Yc + cfg.cam_height, (D, H, W))

    out = np.empty((N, D, H, W, 3), dtype=np.int64)
    for n in range(N):
        psi = math.radians(n * cfg.yaw_step_deg)
        c, s = math.cos(psi), math.sin(psi)
        x = c * x0 - s * y0
        y = s * x0 + c * y0
        out[n, ..., 0] = _floor_index(x, cfg.xy_lo, cfg.xy_res)
        out[n, ..., 1] = _floor_index(y, cfg.xy_lo, cfg.xy_res)
        out[n, ..., 2] = _floor_index(z, cfg.z_lo, cfg.z_res)
    one = out.reshape(-1, 3).astype(np.int32)
    if cfg.B == 1:
        return np.ascontiguousarray(one)
    return np.ascontiguousarray(np.tile(one, (cfg.B, 1)))


def random_coor(rng: np.random.Generator, shape: dict, p_out: float = 0.3,
                spread: int = 2) -> np.ndarray:
    """Random voxel indices for small test shapes.

    Each point draws x, y, z uniformly from an interval that overhangs the
    grid by ``spread`` cells on both sides, so that roughly ``p_out`` of the
    points (tunable through ``spread``) fall outside the grid, including
    negative indices and indices equal to the upper bound.
    """
    B, N, D, H, W = (shape[k] for k in "BNDHW")
    X, Y, Z = shape["X"], shape["Y"], shape["Z"]
    P = B * N * D * H * W
    coor = np.empty((P, 3), dtype=np.int32)
    for col, ext in enumerate((X, Y, Z)):
        coor[:, col] = rng.integers(-spread, ext + spread, size=P)
    # Force a fraction of points inside the grid so the test is not all-empty.
    inside = rng.random(P) >= p_out
    for col, ext in enumerate((X, Y, Z)):
        coor[inside, col] = rng.integers(0, ext, size=int(inside.sum()))
    return coor


# ---- the rig as camera parameters (for the on-device geometry) -------------
#
# Per camera, 16 float64 values: fx, fy, cx, cy, then the camera-to-ego
# rotation R (row-major 3x3) and translation t (ego = R @ cam + t).  The
# rig's axis change and yaw above are R = Yaw(psi) @ A with A taking
# (Xc, Yc, Zc) to (Zc, -Xc, -Yc), and t = (0, 0, cam_height).

CAM_WORDS = 16


def rig_cameras(cfg: Config) -> np.ndarray:
    """float64 (B, N, 16): every sample's camera parameters of the rig."""
    f = cfg.focal
    cams = np.zeros((cfg.N, CAM_WORDS), dtype=np.float64)
    for n in range(cfg.N):
        psi = math.radians(n * cfg.yaw_step_deg)
        c, s = math.cos(psi), math.sin(psi)
        R = np.array([[s, 0.0, c], [-c, 0.0, s], [0.0, -1.0, 0.0]])
        cams[n, :4] = (f, f, cfg.img_w / 2.0, cfg.img_h / 2.0)
        cams[n, 4:13] = R.reshape(-1)
        cams[n, 13:16] = (0.0, 0.0, cfg.cam_height)
    return np.ascontiguousarray(np.broadcast_to(cams, (cfg.B, cfg.N, CAM_WORDS)))


def frustum_params(cfg: Config) -> dict:
    """The frustum and grid description the geometry takes."""
    return dict(stride=float(cfg.stride), depth_start=float(cfg.depth_start),
                depth_step=float(cfg.depth_step),
                lo=(float(cfg.xy_lo), float(cfg.xy_lo), float(cfg.z_lo)),
                res=(float(cfg.xy_res), float(cfg.xy_res), float(cfg.z_res)))


def jittered_cameras(cfg: Config, rng: np.random.Generator, yaw_deg: float = 5.0,
                     shift_m: float = 0.5) -> np.ndarray:
    """The rig with an independent random yaw (up to +-yaw_deg) and ego
    shift (up to +-shift_m in x and y) per sample: per-sample augmentation."""
    cams = rig_cameras(cfg).copy()
    for b in range(cfg.B):
        dpsi = math.radians(rng.uniform(-yaw_deg, yaw_deg))
        c, s = math.cos(dpsi), math.sin(dpsi)
        Y = np.array([[c, -s, 0.0], [s, c, 0.0], [0.0, 0.0, 1.0]])
        dx, dy = rng.uniform(-shift_m, shift_m, size=2)
        for n in range(cfg.N):
            R = cams[b, n, 4:13].reshape(3, 3)
            cams[b, n, 4:13] = (Y @ R).reshape(-1)
            t = cams[b, n, 13:16]
            cams[b, n, 13:16] = Y @ t + np.array([dx, dy, 0.0])
    return cams

"""The five synthetic workloads, shaped like the paper's view-transform runs.

BEVPoolv2 (section 2.1 and Fig. 2) times the view transformation on six
surround cameras with stride-16 feature maps at input resolutions from
256x704 to 640x1760, with D=59 or D=118 depth classes, pooling into a
128x128 BEV grid at 0.8 m.  The paper uses nuScenes calibrations; none are
available here, so an idealised rig stands in: six pinhole cameras 60 deg
apart in yaw, 70 deg horizontal field of view, mounted 1.5 m above the ego
origin with no pitch or roll.  The BEV grid is centred on the ego origin
(section 2.3 moves the receptive field to the ego frame).
"""

from __future__ import annotations

import math
from dataclasses import dataclass


@dataclass(frozen=True)
class Config:
    name: str
    B: int                 # samples sharing one camera rig
    N: int                 # camera views
    img_h: int             # input image height in pixels
    img_w: int             # input image width in pixels
    stride: int            # feature-map stride
    D: int                 # depth classes
    depth_start: float     # metres, first depth bin
    depth_step: float      # metres between depth bins
    C: int                 # feature channels
    dtype: str             # "f32" or "f16": depth score and feature
    out_dtype: str         # "f32" or "f16": BEV output and its gradient
    xy_lo: float           # BEV grid lower bound in x and y (metres)
    xy_hi: float           # BEV grid upper bound in x and y (metres, exclusive)
    xy_res: float          # BEV cell size in x and y (metres)
    z_lo: float = -5.0
    z_hi: float = 3.0
    z_res: float = 8.0
    hfov_deg: float = 70.0
    cam_height: float = 1.5
    yaw_step_deg: float = 60.0
    seed: int = 0
    backward: bool = True  # whether the workload exercises the backward pass

    # --- derived sizes -------------------------------------------------
    @property
    def H(self) -> int:
        return self.img_h // self.stride

    @property
    def W(self) -> int:
        return self.img_w // self.stride

    @property
    def X(self) -> int:
        return int(round((self.xy_hi - self.xy_lo) / self.xy_res))

    @property
    def Y(self) -> int:
        return self.X

    @property
    def Z(self) -> int:
        return int(round((self.z_hi - self.z_lo) / self.z_res))

    @property
    def P(self) -> int:
        """Frustum points B*N*D*H*W."""
        return self.B * self.N * self.D * self.H * self.W

    @property
    def cells(self) -> int:
        """BEV cells B*Z*Y*X."""
        return self.B * self.Z * self.Y * self.X

    @property
    def focal(self) -> float:
        return (self.img_w / 2.0) / math.tan(math.radians(self.hfov_deg) / 2.0)

    def shape(self) -> dict:
        return dict(B=self.B, N=self.N, D=self.D, H=self.H, W=self.W,
                    C=self.C, X=self.X, Y=self.Y, Z=self.Z)


CONFIGS: dict[str, Config] = {
    # 1 camera, 4x8 feature map, 8 depth bins, 16x16 BEV at 1 m.
    "tiny": Config(name="tiny", B=1, N=1, img_h=64, img_w=128, stride=16,
                   D=8, depth_start=1.0, depth_step=1.0, C=16,
                   dtype="f32", out_dtype="f32",
                   xy_lo=-8.0, xy_hi=8.0, xy_res=1.0, seed=0),
    # BEVDet-R50 shape: 256x704 input, D=59 (1..59 m), C=64.
    "bevdet": Config(name="bevdet", B=1, N=6, img_h=256, img_w=704, stride=16,
                     D=59, depth_start=1.0, depth_step=1.0, C=64,
                     dtype="f32", out_dtype="f32",
                     xy_lo=-51.2, xy_hi=51.2, xy_res=0.8, seed=1),
    # Headline shape of the abstract: 640x1600 input, D=118 (1..59.5 m step 0.5), C=80.
    "headline": Config(name="headline", B=1, N=6, img_h=640, img_w=1600, stride=16,
                       D=118, depth_start=1.0, depth_step=0.5, C=80,
                       dtype="f32", out_dtype="f32",
                       xy_lo=-51.2, xy_hi=51.2, xy_res=0.8, seed=2,
                       backward=False),
    # Four samples at 640x1760, fp16 depth/feature, 256x256 BEV at 0.4 m.
    "large": Config(name="large", B=4, N=6, img_h=640, img_w=1760, stride=16,
                    D=118, depth_start=1.0, depth_step=0.5, C=80,
                    dtype="f16", out_dtype="f16",
                    xy_lo=-51.2, xy_hi=51.2, xy_res=0.4, seed=3),
    # The headline rig into a 3-D voxel grid: z over [-5, 3) m in 0.5 m
    # slices, so 128x128x16 cells.
    "voxel3d": Config(name="voxel3d", B=1, N=6, img_h=640, img_w=1600, stride=16,
                      D=118, depth_start=1.0, depth_step=0.5, C=80,
                      dtype="f32", out_dtype="f32",
                      xy_lo=-51.2, xy_hi=51.2, xy_res=0.8, z_res=0.5, seed=5),
    # Training batch: eight samples at 256x704, D=118, C=80.
    "train": Config(name="train", B=8, N=6, img_h=256, img_w=704, stride=16,
                    D=118, depth_start=1.0, depth_step=0.5, C=80,
                    dtype="f32", out_dtype="f32",
                    xy_lo=-51.2, xy_hi=51.2, xy_res=0.8, seed=4),
}


def get_config(name: str) -> Config:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; choose one of {sorted(CONFIGS)}")

"""Pins for the synthetic rig geometry and activation draws (CPU only)."""

import math

import numpy as np
import pytest

from workloads import CONFIGS, draw_inputs, frustum_coor


def test_config_sizes():
    t = CONFIGS["tiny"]
    assert (t.H, t.W, t.X, t.Y, t.Z, t.P) == (4, 8, 16, 16, 1, 256)
    h = CONFIGS["headline"]
    assert (h.H, h.W, h.X, h.Z, h.P) == (40, 100, 128, 1, 2_832_000)
    assert CONFIGS["large"].X == 256 and CONFIGS["large"].P == 12_460_800
    assert CONFIGS["train"].P == 3_987_456
    assert CONFIGS["bevdet"].P == 249_216
    v = CONFIGS["voxel3d"]
    assert (v.X, v.Y, v.Z, v.P, v.cells) == (128, 128, 16, 2_832_000, 262_144)


def test_voxel3d_height_slices():
    """Camera 0, feature row h = 19 (centre v = 312 px, 8 px above the
    principal point at 320): a ray at elevation atan(8 / f) climbs from
    1.5 m by 8/f per metre of depth, f = 800 / tan(35 deg) = 1142.5 px; over
    1..59.5 m that stays in [1.5, 1.92] m, inside the slice [1.5, 2.0) m,
    index floor((z + 5) / 0.5) = 13.  Row h = 20 (8 px below) descends from
    1.5 m into [1.08, 1.5) m, index 12."""
    cfg = CONFIGS["voxel3d"]
    per_view = cfg.D * cfg.H * cfg.W
    c = frustum_coor(cfg)[:per_view].reshape(cfg.D, cfg.H, cfg.W, 3)
    ext = np.array([cfg.X, cfg.Y, cfg.Z])
    inside = np.all((c >= 0) & (c < ext), axis=-1)
    for h, iz in ((19, 13), (20, 12)):
        kept = inside[:, h, :]
        assert kept.any()
        assert np.all(c[:, h, :, 2][kept] == iz), (h, np.unique(c[:, h, :, 2][kept]))
    # points inside the grid fill all 16 slices
    zs = c[..., 2][inside]
    assert np.array_equal(np.unique(zs), np.arange(16))


def test_hand_evaluated_point_tiny():
    # Camera 0, depth bin 0 (1 m), feature cell h=0, w=0 of the 64x128 image:
    # u = 8, v = 8, cx = 64, cy = 32, f = 64 / tan(35 deg) = 91.4017...
    # ego x = 1 -> ix = floor(1 + 8) = 9
    # ego y = 56/f = 0.6127 -> iy = floor(8.6127) = 8
    # ego z = 1.5 + 24/f = 1.7626 -> iz = floor(6.7626 / 8) = 0
    coor = frustum_coor(CONFIGS["tiny"])
    assert coor[0].tolist() == [9, 8, 0]
    # w = 7 mirrors w = 0 about the optical axis: y = -0.6127 -> iy = 7
    assert coor[7].tolist() == [9, 7, 0]


def test_camera0_depth_is_ego_x():
    # With zero yaw the ego x coordinate equals the depth exactly, so
    # ix = depth - x_lo (integers for the 1 m grid of the tiny rig).
    cfg = CONFIGS["tiny"]
    coor = frustum_coor(cfg).reshape(cfg.D, cfg.H, cfg.W, 3)
    for d in range(cfg.D):
        assert np.all(coor[d, :, :, 0] == d + 1 + 8)


@pytest.mark.parametrize("name", ["tiny", "headline"])
def test_mirror_symmetry_camera0(name):
    cfg = CONFIGS[name]
    per_view = cfg.D * cfg.H * cfg.W
    c = frustum_coor(cfg)[:per_view].reshape(cfg.D, cfg.H, cfg.W, 3)
    iy = c[..., 1]
    mirrored = iy + iy[:, :, ::-1]
    # u_w - cx is antisymmetric in w, so y(w) = -y(W-1-w); away from cell edges
    # the two indices add up to Y - 1.
    assert np.mean(mirrored == cfg.Y - 1) > 0.99
    assert np.array_equal(c[..., 0], c[:, :, ::-1, 0])


def test_opposite_camera_is_point_reflection():
    cfg = CONFIGS["headline"]
    per_view = cfg.D * cfg.H * cfg.W
    c = frustum_coor(cfg)
    cam0 = c[:per_view]
    cam3 = c[3 * per_view:4 * per_view]   # yaw 180 deg: (x, y) -> (-x, -y)
    inside = (cam0[:, 0] >= 0) & (cam0[:, 0] < cfg.X) & (cam0[:, 1] >= 0) & (cam0[:, 1] < cfg.Y)
    # floor(-t) = -floor(t) - 1 except when t sits exactly on a cell edge
    # (camera 0 puts ego x = depth on many edges), where the index moves by one.
    dx = cam3[inside, 0] - (cfg.X - 1 - cam0[inside, 0])
    dy = cam3[inside, 1] - (cfg.Y - 1 - cam0[inside, 1])
    assert np.all((dx == 0) | (dx == 1)) and np.all((dy == 0) | (dy == 1))
    assert np.mean((dx == 0) & (dy == 0)) > 0.8
    assert np.array_equal(cam3[:, 2], cam0[:, 2])


def test_batch_shares_geometry():
    cfg = CONFIGS["train"]
    c = frustum_coor(cfg)
    per_b = cfg.P // cfg.B
    assert np.array_equal(c[:per_b], c[per_b:2 * per_b])


def test_draws_are_seeded_and_shaped():
    cfg = CONFIGS["tiny"]
    a = draw_inputs(cfg)
    b = draw_inputs(cfg)
    assert np.array_equal(a["depth"], b["depth"]) and np.array_equal(a["feat"], b["feat"])
    assert a["depth"].shape == (1, 1, 8, 4, 8) and a["feat"].shape == (1, 1, 4, 8, 16)
    assert a["grad_out"].shape == (1, 1, 16, 16, 16)
    s = a["depth"].astype(np.float64).sum(axis=2)
    assert np.allclose(s, 1.0, atol=1e-6)
    assert a["depth"].dtype == np.float32


def test_fp16_draws():
    cfg = CONFIGS["large"]
    small = cfg.__class__(**{**cfg.__dict__, "B": 1, "img_h": 64, "img_w": 128})
    d = draw_inputs(small)
    assert d["depth"].dtype == np.float16 and d["feat"].dtype == np.float16
    assert d["grad_out"].dtype == np.float16

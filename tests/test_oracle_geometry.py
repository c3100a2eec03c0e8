"""Pins of the oracle's voxel index from camera parameters (CPU only).

oracle.geometry_ref is the general pinhole form (intrinsics, a camera-to-ego
rotation and translation, floor of the grid coordinate).  The rig in
workloads/rig.py computes the same indices by its own route: an explicit
axis change and yaw, with no matrix.  Fed the rig's cameras, the oracle
must give the rig's indices bit for bit on every workload; a hand-evaluated
point and planted mistakes pin it further.
"""

import math

import numpy as np
import pytest

import oracle
from workloads import CONFIGS, frustum_coor, frustum_params, jittered_cameras, rig_cameras


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_matches_the_rig_bit_for_bit(name):
    cfg = CONFIGS[name]
    got = oracle.geometry_ref(rig_cameras(cfg), frustum_params(cfg), cfg.shape())
    assert got.dtype == np.int32 and got.shape == (cfg.P, 3)
    assert np.array_equal(got, frustum_coor(cfg))


def test_hand_evaluated_point():
    # tiny, camera 0, bin 0 (1 m), cell (0, 0): u = v = 8, cx = 64, cy = 32,
    # f = 64 / tan(35 deg): ego (1, 56/f, 1.5 + 24/f) -> (9, 8, 0)
    cfg = CONFIGS["tiny"]
    g = oracle.geometry_ref(rig_cameras(cfg), frustum_params(cfg), cfg.shape())
    assert g[0].tolist() == [9, 8, 0]
    f = 64 / math.tan(math.radians(35))
    assert math.floor(56 / f + 8) == 8 and math.floor((1.5 + 24 / f + 5) / 8) == 0


def test_per_sample_cameras_move_the_points():
    """Each sample takes its own cameras: a sample's indices depend only on
    its own parameters."""
    cfg = CONFIGS["train"]
    rng = np.random.default_rng(3)
    cams = jittered_cameras(cfg, rng)
    g = oracle.geometry_ref(cams, frustum_params(cfg), cfg.shape()).reshape(cfg.B, -1, 3)
    for b in range(cfg.B):
        one = oracle.geometry_ref(cams[b:b + 1], frustum_params(cfg), dict(cfg.shape(), B=1))
        assert np.array_equal(g[b], one)
    assert not np.array_equal(g[0], g[1])


def test_planted_mistakes_caught():
    cfg = CONFIGS["bevdet"]
    cams = rig_cameras(cfg)
    want = frustum_coor(cfg)
    p = frustum_params(cfg)
    transposed = cams.copy()
    transposed[..., 4:13] = cams[..., 4:13].reshape(cfg.B, cfg.N, 3, 3).transpose(0, 1, 3, 2).reshape(cfg.B, cfg.N, 9)
    assert not np.array_equal(oracle.geometry_ref(transposed, p, cfg.shape()), want)
    swapped = cams.copy()
    swapped[..., 2], swapped[..., 3] = cams[..., 3], cams[..., 2]  # cx <-> cy
    assert not np.array_equal(oracle.geometry_ref(swapped, p, cfg.shape()), want)
    q = dict(p, depth_start=p["depth_start"] + p["depth_step"])  # off by one depth bin
    assert not np.array_equal(oracle.geometry_ref(cams, q, cfg.shape()), want)

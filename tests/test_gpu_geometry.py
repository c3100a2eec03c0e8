"""On-device geometry against the oracle, bit for bit (section 2.1: each
frustum point's voxel index from the camera intrinsics and extrinsics).

The indices are integers decided by float64 arithmetic that both sides take
in the same order, so they must agree exactly: on every workload's rig, on
per-sample jittered cameras (augmentation), and through the whole path -
geometry, then prepare, whose plan must equal the oracle's plan of the
oracle's indices.
"""

import numpy as np
import pytest
import torch

import _gpu
import oracle
from paper_2211_17111_amd import bevpool as bp
from workloads import CONFIGS, frustum_params, jittered_cameras, rig_cameras

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "bevdet", "headline", "large", "train", "voxel3d"])
def test_rig_geometry_bit_exact(name):
    cfg = CONFIGS[name]
    _gpu.say(f"geometry: {name}")
    cams = rig_cameras(cfg)
    got = bp.geometry(torch.from_numpy(cams).to(_gpu.DEV), frustum_params(cfg), cfg.shape())
    torch.cuda.synchronize()
    want = oracle.geometry_ref(cams, frustum_params(cfg), cfg.shape())
    assert np.array_equal(got.cpu().numpy(), want), name


def test_jittered_geometry_then_prepare():
    """Per-sample cameras (augmentation): the device geometry, then the
    device prepare, against the oracle's geometry and plan."""
    cfg = CONFIGS["train"]
    shape = cfg.shape()
    cams = jittered_cameras(cfg, np.random.default_rng(8))
    coor_d = bp.geometry(torch.from_numpy(cams).to(_gpu.DEV), frustum_params(cfg), shape)
    torch.cuda.synchronize()
    want = oracle.geometry_ref(cams, frustum_params(cfg), shape)
    assert np.array_equal(coor_d.cpu().numpy(), want)
    plan = bp.prepare(coor_d, shape)
    ref = oracle.prepare_ref(want, shape)
    assert (plan.n_valid, plan.n_intervals) == (ref["n_valid"], ref["n_intervals"])
    nv, ni = plan.n_valid, plan.n_intervals
    for k in ("ranks_depth", "ranks_feat", "ranks_bev"):
        assert np.array_equal(getattr(plan, k)[:nv].cpu().numpy(), ref[k][:nv]), k
    assert np.array_equal(plan.interval_starts[:ni].cpu().numpy(), ref["interval_starts"][:ni])
    assert np.array_equal(plan.interval_lengths[:ni].cpu().numpy(), ref["interval_lengths"][:ni])


@pytest.mark.parametrize("dhw", [(3, 1, 1), (5, 1, 257), (2, 17, 15), (130, 2, 3)])
def test_geometry_ragged_shapes(dhw):
    """Views of one pixel, of 257 pixels (a block and one more), of an odd
    pixel count, and of more depth bins than pixels: the grid covers each
    view's pixels in blocks, its depth bins and its views."""
    cfg = CONFIGS["tiny"]
    D, H, W = dhw
    shape = dict(cfg.shape(), D=D, H=H, W=W)
    _gpu.say(f"geometry ragged shape D={D} H={H} W={W}")
    cams = rig_cameras(cfg)
    got = bp.geometry(torch.from_numpy(cams).to(_gpu.DEV), frustum_params(cfg), shape)
    torch.cuda.synchronize()
    want = oracle.geometry_ref(cams, frustum_params(cfg), shape)
    assert np.array_equal(got.cpu().numpy(), want), dhw

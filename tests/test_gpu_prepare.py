"""GPU prepare (filter, radix sort, intervals) is bit-exact with the oracle."""

import numpy as np
import pytest

import _gpu
import oracle
from workloads import CONFIGS, frustum_coor, random_coor

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "bevdet", "headline", "large", "train", "voxel3d"])
def test_prepare_configs(name):
    cfg = CONFIGS[name]
    _gpu.say(f"prepare parity: {name} P={cfg.P}")
    coor = frustum_coor(cfg)
    got = _gpu.plan_to_numpy(_gpu.run_prepare(coor, cfg.shape()))
    _gpu.assert_plan_equal(got, oracle.prepare_ref(coor, cfg.shape()), name)


# Shapes chosen to span several 1024-point tiles with ragged tails, one to
# three radix passes (key bits 1..21), B > 1, and interval chunks of one to
# two 1024-cell parts (the last shape has 2^21 cells).
RANDOM_SHAPES = [
    dict(B=1, N=1, D=1, H=1, W=1, C=4, X=1, Y=1, Z=1),          # P = 1, one cell
    dict(B=1, N=1, D=3, H=5, W=7, C=4, X=3, Y=2, Z=1),          # P = 105
    dict(B=2, N=3, D=11, H=13, W=17, C=8, X=40, Y=30, Z=2),     # P = 14586, 4 tiles + tail
    dict(B=3, N=2, D=7, H=9, W=100, C=8, X=256, Y=256, Z=1),    # 18-bit keys, 3 passes
    dict(B=1, N=6, D=5, H=16, W=44, C=64, X=512, Y=300, Z=1),   # 18 bits
    dict(B=1, N=1, D=2, H=40, W=50, C=4, X=1024, Y=1024, Z=2),  # 21 bits, 2^21 cells
]


@pytest.mark.parametrize("k", range(len(RANDOM_SHAPES)))
def test_prepare_random(k):
    shape = RANDOM_SHAPES[k]
    rng = np.random.default_rng(100 + k)
    coor = random_coor(rng, shape)
    _gpu.say(f"prepare random shape {shape}")
    got = _gpu.plan_to_numpy(_gpu.run_prepare(coor, shape))
    _gpu.assert_plan_equal(got, oracle.prepare_ref(coor, shape), str(shape))


def test_prepare_edge_cases():
    shape = dict(B=2, N=1, D=4, H=30, W=50, C=4, X=16, Y=16, Z=2)   # P = 12000
    P = 12000
    rng = np.random.default_rng(0)
    cases = {
        "nothing in range": np.full((P, 3), -1, dtype=np.int32),
        "all in one cell": np.tile(np.array([[3, 5, 1]], dtype=np.int32), (P, 1)),
        "single kept point": np.concatenate([np.full((P - 1, 3), 99, dtype=np.int32),
                                             np.array([[15, 15, 1]], dtype=np.int32)]),
        "exactly on the bounds": np.stack([rng.choice([-1, 0, 15, 16], P),
                                           rng.choice([-1, 0, 15, 16], P),
                                           rng.choice([-1, 0, 1, 2], P)], axis=1).astype(np.int32),
        "huge and negative indices": np.stack([rng.integers(-2**31, 2**31 - 1, P),
                                               rng.integers(-2**31, 2**31 - 1, P),
                                               rng.integers(0, 2, P)], axis=1).astype(np.int32),
    }
    # kept counts at and beside a later-pass tile boundary (1024 points): the
    # later passes histogram and scan only the tiles holding kept points
    for kept in (1023, 1024, 1025, 2048, 2049):
        coor = np.full((P, 3), 99, dtype=np.int32)
        idx = np.sort(rng.choice(P, kept, replace=False))
        coor[idx] = np.stack([rng.integers(0, 16, kept), rng.integers(0, 16, kept),
                              rng.integers(0, 2, kept)], axis=1)
        cases[f"{kept} kept points"] = coor
    for label, coor in cases.items():
        _gpu.say(f"prepare edge case: {label}")
        got = _gpu.plan_to_numpy(_gpu.run_prepare(coor, shape))
        _gpu.assert_plan_equal(got, oracle.prepare_ref(coor, shape), label)


def test_prepare_unaligned_coor():
    """coor at a 4-byte offset from a 16-byte boundary takes the scalar loads;
    the result is the same plan."""
    import torch
    from paper_2211_17111_amd import bevpool as bp
    cfg = CONFIGS["bevdet"]
    coor = frustum_coor(cfg)
    _gpu.say("prepare with coor at a 4-byte offset")
    flat = torch.empty(coor.size + 1, dtype=torch.int32, device=_gpu.DEV)
    flat[1:].copy_(torch.from_numpy(coor.reshape(-1)))
    dev_coor = flat[1:].view(coor.shape)
    assert dev_coor.data_ptr() % 16 != 0
    got = _gpu.plan_to_numpy(bp.prepare(dev_coor, cfg.shape()))
    _gpu.assert_plan_equal(got, oracle.prepare_ref(coor, cfg.shape()), "unaligned coor")


def test_prepare_deterministic():
    cfg = CONFIGS["bevdet"]
    coor = frustum_coor(cfg)
    a = _gpu.plan_to_numpy(_gpu.run_prepare(coor, cfg.shape()))
    b = _gpu.plan_to_numpy(_gpu.run_prepare(coor, cfg.shape()))
    _gpu.assert_plan_equal(a, b, "rerun")

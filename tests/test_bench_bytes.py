"""The algorithmic byte counts that bench.py divides by (CPU only).

Forward: depth of kept points, the feature tensor once, two ranks per kept
point, the interval table and every output element once.  Backward: the
occupied cells' grad_out rows, the feature tensor, depth of kept points, the
ranks and interval table, all of grad_depth and all of grad_feat.  Checked
against the per-workload figures of the measurement plan (forward 6.95 /
29.84 / 125.5 / 78.6 MB for BEVDet / headline / large / train, backward
95.3 MB for train), from the kept-point and interval counts of the oracle's
plan for those workloads.
"""

import importlib.util
import os

import pytest

from workloads import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# kept points and occupied cells of the oracle's plan
COUNTS = {"bevdet": (130160, 9681), "headline": (1393712, 15648), "large": (6452336, 176056),
          "train": (2057728, 99440)}


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name,mb", [("bevdet", 6.95), ("headline", 29.84), ("large", 125.48),
                                     ("train", 78.64)])
def test_forward_bytes(name, mb):
    b = _bench()
    assert round(b.forward_min_bytes(CONFIGS[name], *COUNTS[name]) / 1e6, 2) == mb


def test_backward_bytes_train():
    b = _bench()
    assert round(b.backward_min_bytes(CONFIGS["train"], *COUNTS["train"]) / 1e6, 1) == 95.3


def test_prepare_bytes_headline():
    # the voxel index (x, y, z) of every frustum point read once, three ranks per
    # kept point and the interval table (start, length) written once, plus the counts
    b = _bench()
    cfg = CONFIGS["headline"]
    nv, ni = COUNTS["headline"]
    assert b.prepare_min_bytes(cfg, nv, ni) == 3 * 4 * cfg.P + 3 * 4 * nv + 2 * 4 * ni + 2 * 4

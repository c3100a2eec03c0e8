"""The CPU oracle against brute force, closed forms and a hand-worked example.

These tests run without a GPU.  They pin ``oracle/`` to the paper's
definition (BEVPoolv2 section 2.1) through routes that share none of its
code; see ``_pins.py``.
"""

import json
import os

import numpy as np
import pytest

import _pins
import oracle
from workloads import CONFIGS, draw_inputs, draw_small, frustum_coor, random_coor

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SMALL_SHAPES = [
    dict(B=1, N=1, D=3, H=2, W=3, C=4, X=3, Y=4, Z=1),
    dict(B=2, N=2, D=4, H=2, W=3, C=5, X=4, Y=3, Z=2),
    dict(B=3, N=1, D=2, H=3, W=2, C=1, X=2, Y=2, Z=3),
]


def _tiny():
    cfg = CONFIGS["tiny"]
    return cfg, cfg.shape(), frustum_coor(cfg), draw_inputs(cfg)


# --------------------------------------------------------------- hand example

def _hand():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        g = json.load(f)
    s = g["shape"]
    coor = np.array(g["coor"], dtype=np.int32)
    depth = np.array(g["depth"], dtype=np.float64).reshape(s["B"], s["N"], s["D"], s["H"], s["W"])
    feat = np.array(g["feat"], dtype=np.float64).reshape(s["B"], s["N"], s["H"], s["W"], s["C"])
    grad = np.array(g["grad_out"], dtype=np.float64).reshape(s["B"], s["Z"], s["Y"], s["X"], s["C"])
    return s, coor, depth, feat, grad, g["expected"]


def test_hand_example_prepare():
    s, coor, depth, feat, grad, exp = _hand()
    got = oracle.prepare_ref(coor, s)
    for k in ("ranks_depth", "ranks_feat", "ranks_bev", "interval_starts", "interval_lengths"):
        assert got[k].tolist() == exp[k], k
    assert got["n_valid"] == exp["n_valid"]
    assert got["n_intervals"] == exp["n_intervals"]


def test_hand_example_forward_backward():
    s, coor, depth, feat, grad, exp = _hand()
    out, _ = oracle.forward_ref(depth, feat, coor, s)
    assert out.reshape(-1, s["C"]).tolist() == exp["out"]
    gd, gf, _, _ = oracle.backward_ref(grad, depth, feat, coor, s)
    assert gd.reshape(-1).tolist() == exp["grad_depth"]
    assert gf.reshape(-1, s["C"]).tolist() == exp["grad_feat"]


# ------------------------------------------------------------------- prepare

def test_prepare_brute_tiny():
    cfg, shape, coor, _ = _tiny()
    assert _pins.check_prepare_brute(oracle.prepare_ref, coor, shape) == []


@pytest.mark.parametrize("shape", SMALL_SHAPES)
def test_prepare_brute_random(shape):
    rng = np.random.default_rng(11)
    coor = random_coor(rng, shape)
    assert _pins.check_prepare_brute(oracle.prepare_ref, coor, shape) == []


@pytest.mark.parametrize("name", ["tiny", "bevdet", "headline"])
def test_prepare_invariants_configs(name):
    cfg = CONFIGS[name]
    coor = frustum_coor(cfg)
    assert _pins.check_prepare_invariants(oracle.prepare_ref, coor, cfg.shape()) == []


def test_prepare_counts_match_independent_probe():
    # Counts computed by an independent throwaway script under the same rig
    # conventions: (n_valid, n_intervals, longest interval).
    probe = {"tiny": (208, 40, 16), "bevdet": (130160, 9681, 528),
             "headline": (1393712, 15648, 4520), "train": (2057728, 99440, 800)}
    for name, (nv, ni, mx) in probe.items():
        cfg = CONFIGS[name]
        got = oracle.prepare_ref(frustum_coor(cfg), cfg.shape())
        assert (got["n_valid"], got["n_intervals"], int(got["interval_lengths"].max())) == (nv, ni, mx), name


def test_prepare_edge_cases():
    shape = dict(B=1, N=1, D=2, H=2, W=2, C=3, X=2, Y=2, Z=1)
    P = 8
    # nothing in range
    coor = np.full((P, 3), -1, dtype=np.int32)
    got = oracle.prepare_ref(coor, shape)
    assert got["n_valid"] == 0 and got["n_intervals"] == 0
    assert _pins.check_prepare_brute(oracle.prepare_ref, coor, shape) == []
    # all points in one cell
    coor = np.zeros((P, 3), dtype=np.int32)
    got = oracle.prepare_ref(coor, shape)
    assert got["interval_lengths"].tolist() == [P]
    assert got["ranks_depth"].tolist() == list(range(P))
    # exactly on the upper bounds -> dropped; one below -> kept
    coor = np.array([[2, 0, 0], [0, 2, 0], [0, 0, 1], [1, 1, 0],
                     [-1, 0, 0], [0, -1, 0], [0, 0, -1], [1, 0, 0]], dtype=np.int32)
    got = oracle.prepare_ref(coor, shape)
    assert got["ranks_depth"].tolist() == [7, 3]
    assert got["ranks_bev"].tolist() == [1, 3]


# ------------------------------------------------------------------- forward

def test_forward_brute_tiny():
    cfg, shape, coor, data = _tiny()
    assert _pins.check_forward_brute(oracle.forward_ref, data["depth"], data["feat"], coor, shape) == []


@pytest.mark.parametrize("shape", SMALL_SHAPES)
def test_forward_brute_random(shape):
    rng = np.random.default_rng(5)
    coor = random_coor(rng, shape)
    data = draw_small(rng, shape)
    assert _pins.check_forward_brute(oracle.forward_ref, data["depth"], data["feat"], coor, shape) == []


@pytest.mark.parametrize("shape", SMALL_SHAPES)
def test_forward_identities_random(shape):
    rng = np.random.default_rng(6)
    coor = random_coor(rng, shape)
    data = draw_small(rng, shape, softmax=False)
    assert _pins.check_forward_identities(oracle.forward_ref, data["depth"], data["feat"], coor, shape) == []


def test_forward_identities_tiny_and_fp16():
    cfg, shape, coor, data = _tiny()
    assert _pins.check_forward_identities(oracle.forward_ref, data["depth"], data["feat"], coor, shape) == []
    d16 = data["depth"].astype(np.float16)
    f16 = data["feat"].astype(np.float16)
    assert _pins.check_forward_brute(oracle.forward_ref, d16, f16, coor, shape) == []


def test_forward_empty_cells_exactly_zero():
    cfg, shape, coor, data = _tiny()
    out, _ = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    prep = oracle.prepare_ref(coor, shape)
    occupied = np.zeros(cfg.cells, dtype=bool)
    occupied[prep["ranks_bev"]] = True
    flat = out.reshape(cfg.cells, -1)
    assert np.all(flat[~occupied] == 0.0)
    assert np.all(np.any(flat[occupied] != 0.0, axis=1))


# ------------------------------------------------------------------ backward

def test_backward_brute_tiny():
    cfg, shape, coor, data = _tiny()
    assert _pins.check_backward_brute(oracle.backward_ref, data["grad_out"], data["depth"],
                                      data["feat"], coor, shape) == []


@pytest.mark.parametrize("shape", SMALL_SHAPES)
def test_backward_brute_random(shape):
    rng = np.random.default_rng(8)
    coor = random_coor(rng, shape)
    data = draw_small(rng, shape)
    assert _pins.check_backward_brute(oracle.backward_ref, data["grad_out"], data["depth"],
                                      data["feat"], coor, shape) == []


@pytest.mark.parametrize("shape", SMALL_SHAPES)
def test_backward_identities_random(shape):
    rng = np.random.default_rng(9)
    coor = random_coor(rng, shape)
    data = draw_small(rng, shape)
    assert _pins.check_backward_identities(oracle.backward_ref, oracle.forward_ref, data["grad_out"],
                                           data["depth"], data["feat"], coor, shape) == []


def test_backward_identities_tiny():
    cfg, shape, coor, data = _tiny()
    assert _pins.check_backward_identities(oracle.backward_ref, oracle.forward_ref, data["grad_out"],
                                           data["depth"], data["feat"], coor, shape) == []


# ------------------------------------------------------------- sampled forms

@pytest.mark.parametrize("name", ["tiny", "bevdet"])
def test_sampled_forms_match_full(name):
    cfg = CONFIGS[name]
    shape = cfg.shape()
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    rng = np.random.default_rng(3)
    out, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    cells = rng.choice(cfg.cells, size=min(64, cfg.cells), replace=False)
    o, m = oracle.forward_cells_ref(data["depth"], data["feat"], coor, shape, cells)
    assert np.allclose(o, out.reshape(cfg.cells, -1)[cells], rtol=0, atol=1e-12)
    assert np.allclose(m, mag.reshape(cfg.cells, -1)[cells], rtol=0, atol=1e-12)
    gd, gf, gdm, gfm = oracle.backward_ref(data["grad_out"], data["depth"], data["feat"], coor, shape)
    pts = rng.choice(cfg.P, size=min(200, cfg.P), replace=False)
    v, m = oracle.grad_depth_points_ref(data["grad_out"], data["feat"], coor, shape, pts)
    assert np.allclose(v, gd.reshape(-1)[pts], rtol=0, atol=1e-12)
    assert np.allclose(m, gdm.reshape(-1)[pts], rtol=0, atol=1e-12)
    rows = cfg.B * cfg.N * cfg.H * cfg.W
    pix = rng.choice(rows, size=min(50, rows), replace=False)
    v, m = oracle.grad_feat_pixels_ref(data["grad_out"], data["depth"], coor, shape, pix)
    assert np.allclose(v, gf.reshape(rows, -1)[pix], rtol=0, atol=1e-12)
    assert np.allclose(m, gfm.reshape(rows, -1)[pix], rtol=0, atol=1e-12)

"""GPU backward (grad_depth, grad_feat) against the float64 oracle."""

import numpy as np
import pytest
import torch

import _gpu
import oracle
from paper_2211_17111_amd import bevpool as bp
from workloads import CONFIGS, draw_inputs, draw_small, frustum_coor, random_coor

pytestmark = pytest.mark.gpu

PATHS = ["plan", "scheduled"]


@pytest.fixture(params=PATHS)
def path(request):
    return request.param


def _bwd(path, g, d, f, plan):
    if path == "scheduled":
        return bp.backward_scheduled(g, d, f, bp.schedule(plan))
    return bp.backward(g, d, f, plan)


def _run(data, coor, shape, path="plan"):
    plan = _gpu.run_prepare(coor, shape)
    gd, gf = _bwd(path, _gpu.to_dev(data["grad_out"]), _gpu.to_dev(data["depth"]),
                  _gpu.to_dev(data["feat"]), plan)
    torch.cuda.synchronize()
    return gd, gf, plan


@pytest.mark.parametrize("name", ["tiny", "bevdet"])
def test_backward_full(name, path):
    cfg = CONFIGS[name]
    _gpu.say(f"backward full parity: {name} {path}")
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    gd, gf, _ = _run(data, coor, cfg.shape(), path)
    rgd, rgf, mgd, mgf = oracle.backward_ref(data["grad_out"], data["depth"], data["feat"], coor,
                                             cfg.shape())
    _gpu.assert_within(gd.cpu().numpy(), rgd, mgd, cfg.dtype, f"{name} grad_depth")
    _gpu.assert_within(gf.cpu().numpy(), rgf, mgf, cfg.dtype, f"{name} grad_feat")
    kept = oracle.kept_mask(coor, cfg.shape())
    assert np.all(gd.cpu().numpy().reshape(-1)[~kept] == 0.0)


# C picks the pixel kernel's lane-group size and vectors per lane: with 4-wide
# (f32) or 8-wide (f16) vectors where C allows, else scalars, these cover
# groups of 1 to 64 lanes and 1, 2, 4, 8 and 16 vectors per lane
@pytest.mark.parametrize("C", [1, 3, 7, 16, 17, 24, 80, 200, 260, 600, 1023])
@pytest.mark.parametrize("dtype,out_dtype", [("f32", "f32"), ("f16", "f16"), ("f16", "f32")])
def test_backward_random_channels(C, dtype, out_dtype, path):
    shape = dict(B=2, N=2, D=9, H=7, W=13, C=C, X=12, Y=10, Z=2)
    rng = np.random.default_rng(50 + C)
    coor = random_coor(rng, shape, p_out=0.4)
    data = draw_small(rng, shape, dtype=dtype, out_dtype=out_dtype)
    _gpu.say(f"backward random C={C} {dtype}/{out_dtype} {path}")
    gd, gf, _ = _run(data, coor, shape, path)
    rgd, rgf, mgd, mgf = oracle.backward_ref(data["grad_out"], data["depth"], data["feat"], coor, shape)
    _gpu.assert_within(gd.float().cpu().numpy(), rgd, mgd, dtype, f"C={C} grad_depth")
    _gpu.assert_within(gf.float().cpu().numpy(), rgf, mgf, dtype, f"C={C} grad_feat")


def test_backward_edge_cases(path):
    shape = dict(B=1, N=2, D=70, H=6, W=10, C=16, X=4, Y=4, Z=1)   # D > 64 depth chunks
    P = 2 * 70 * 60
    rng = np.random.default_rng(3)
    data = draw_small(rng, shape)
    cases = {
        "no point in range": np.full((P, 3), 9, dtype=np.int32),
        "all points in one cell": np.tile(np.array([[1, 2, 0]], dtype=np.int32), (P, 1)),
        "cells alternating along depth": np.tile(np.array([[1, 2, 0]], dtype=np.int32), (P, 1)),
        "random": random_coor(rng, shape),
    }
    # every point its own pair: 70 pairs per pixel, more than one chunk of a lane group
    cases["cells alternating along depth"].reshape(2, 70, 60, 3)[:, 1::2, :, 0] = 3
    for label, coor in cases.items():
        _gpu.say(f"backward edge case: {label} {path}")
        gd, gf, _ = _run(data, coor, shape, path)
        rgd, rgf, mgd, mgf = oracle.backward_ref(data["grad_out"], data["depth"], data["feat"],
                                                 coor, shape)
        _gpu.assert_within(gd.cpu().numpy(), rgd, mgd, "f32", f"{label} grad_depth")
        _gpu.assert_within(gf.cpu().numpy(), rgf, mgf, "f32", f"{label} grad_feat")


@pytest.mark.parametrize("name", ["headline", "large", "train"])
def test_backward_full_size_sampled(name, path):
    cfg = CONFIGS[name]
    _gpu.say(f"backward sampled parity: {name} {path}")
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    gd, gf, plan = _run(data, coor, cfg.shape(), path)
    rng = np.random.default_rng(11)
    # points: random, plus every point of the longest interval
    st = plan.interval_starts.cpu().numpy()
    ln = plan.interval_lengths.cpu().numpy()
    j = int(np.argmax(ln))
    longest = plan.ranks_depth[st[j]:st[j] + ln[j]].cpu().numpy()[:500]
    pts = np.unique(np.concatenate([rng.choice(cfg.P, 3000, replace=False), longest]))
    v, m = oracle.grad_depth_points_ref(data["grad_out"], data["feat"], coor, cfg.shape(), pts)
    got = gd.reshape(-1)[torch.from_numpy(pts).to(_gpu.DEV)].float().cpu().numpy()
    _gpu.assert_within(got, v, m, cfg.dtype, f"{name} grad_depth")
    rows = cfg.B * cfg.N * cfg.H * cfg.W
    pix = np.unique(np.concatenate([rng.choice(rows, 150, replace=False), [0, rows - 1]]))
    v, m = oracle.grad_feat_pixels_ref(data["grad_out"], data["depth"], coor, cfg.shape(), pix)
    got = gf.reshape(rows, cfg.C)[torch.from_numpy(pix).to(_gpu.DEV)].float().cpu().numpy()
    _gpu.assert_within(got, v, m, cfg.dtype, f"{name} grad_feat")
    # dropped points have exactly zero gradient; adjoint identity over everything
    kept = oracle.kept_mask(coor, cfg.shape())
    gdn = gd.float().cpu().numpy().reshape(-1)
    assert np.all(gdn[~kept] == 0.0)
    out = bp.forward(_gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"]), plan,
                     out_dtype=torch.float32)
    g64 = data["grad_out"].astype(np.float64)
    lhs = float(np.sum(g64 * out.double().cpu().numpy()))
    rhs_d = float(np.sum(gdn.astype(np.float64) * data["depth"].astype(np.float64).reshape(-1)))
    rhs_f = float(np.sum(gf.double().cpu().numpy() * data["feat"].astype(np.float64)))
    # every term of the trilinear sum is bounded by max|g| * |depth| * |feat|
    kept5 = kept.reshape(cfg.B, cfg.N, cfg.D, cfg.H, cfg.W)
    absmass = float(np.einsum("bndhw,bnhwc->", np.abs(data["depth"].astype(np.float64)) * kept5,
                              np.abs(data["feat"].astype(np.float64))))
    scale = float(np.abs(g64).max()) * absmass + 1.0
    tol = {"f32": 1e-5, "f16": 2e-3}[cfg.dtype]
    assert abs(lhs - rhs_d) <= tol * scale, (lhs, rhs_d, scale)
    assert abs(lhs - rhs_f) <= tol * scale, (lhs, rhs_f, scale)


def test_backward_deterministic(path):
    cfg = CONFIGS["train"]
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    gd1, gf1, plan = _run(data, coor, cfg.shape(), path)
    gd2, gf2 = _bwd(path, _gpu.to_dev(data["grad_out"]), _gpu.to_dev(data["depth"]),
                    _gpu.to_dev(data["feat"]), plan)
    assert torch.equal(gd1, gd2) and torch.equal(gf1, gf2)


def test_backward_paths_agree_on_poisoned_outputs():
    """Both backward entry points overwrite every element (NaN-poisoned
    outputs come back finite) and agree to fp32 rounding."""
    cfg = CONFIGS["bevdet"]
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    plan = _gpu.run_prepare(coor, cfg.shape())
    g, d, f = (_gpu.to_dev(data[k]) for k in ("grad_out", "depth", "feat"))
    sched = bp.schedule(plan)
    gd = torch.full_like(d, float("nan"))
    gf = torch.full_like(f, float("nan"))
    bp.bevpool_backward_scheduled(cfg.shape(), bp.BEVPOOL_F32, bp.BEVPOOL_F32, g, d, f, sched.buffer,
                                  sched.buffer.numel(), plan.n_valid, plan.n_intervals, gd, gf)
    torch.cuda.synchronize()
    assert torch.isfinite(gd).all() and torch.isfinite(gf).all()
    gd2, gf2 = bp.backward(g, d, f, plan)
    assert float((gd - gd2).abs().max()) <= 1e-5 * float(gd2.abs().max()) + 1e-6
    assert float((gf - gf2).abs().max()) <= 1e-5 * float(gf2.abs().max()) + 1e-6


@pytest.mark.parametrize("D", [31, 32, 33, 128, 129, 150])
def test_backward_scheduled_dropped_points_poisoned(D):
    """In a small launch the scheduled backward writes the zeros of dropped
    points itself from a mask of the depth bins each pixel's pairs cover, when
    D fits the mask, else through a clearing launch: NaN-poisoned outputs come
    back equal to the oracle on both sides of the mask's word and size limits."""
    shape = dict(B=1, N=1, D=D, H=5, W=6, C=16, X=6, Y=6, Z=1)
    rng = np.random.default_rng(D)
    coor = random_coor(rng, shape, p_out=0.4)
    data = draw_small(rng, shape)
    _gpu.say(f"backward dropped points poisoned: D={D}")
    plan = _gpu.run_prepare(coor, shape)
    sched = bp.schedule(plan)
    g, d, f = (_gpu.to_dev(data[k]) for k in ("grad_out", "depth", "feat"))
    gd = torch.full_like(d, float("nan"))
    gf = torch.full_like(f, float("nan"))
    bp.bevpool_backward_scheduled(shape, bp.BEVPOOL_F32, bp.BEVPOOL_F32, g, d, f, sched.buffer,
                                  sched.buffer.numel(), plan.n_valid, plan.n_intervals, gd, gf)
    torch.cuda.synchronize()
    rgd, rgf, mgd, mgf = oracle.backward_ref(data["grad_out"], data["depth"], data["feat"], coor, shape)
    _gpu.assert_within(gd.cpu().numpy(), rgd, mgd, "f32", f"D={D} grad_depth")
    _gpu.assert_within(gf.cpu().numpy(), rgf, mgf, "f32", f"D={D} grad_feat")


@pytest.mark.parametrize("use_schedule", [False, True])
def test_autograd_wrapper_tiny(use_schedule):
    """bev_pool with a Plan (plan-only paths) or a Schedule (scheduled paths)."""
    cfg = CONFIGS["tiny"]
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    plan = _gpu.run_prepare(coor, cfg.shape())
    depth = _gpu.to_dev(data["depth"]).requires_grad_(True)
    feat = _gpu.to_dev(data["feat"]).requires_grad_(True)
    out = bp.bev_pool(depth, feat, bp.schedule(plan) if use_schedule else plan)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, cfg.shape())
    _gpu.assert_within(out.detach().cpu().numpy(), ref, mag, "f32", "autograd out")
    out.backward(_gpu.to_dev(data["grad_out"]))
    rgd, rgf, mgd, mgf = oracle.backward_ref(data["grad_out"], data["depth"], data["feat"], coor,
                                             cfg.shape())
    _gpu.assert_within(depth.grad.cpu().numpy(), rgd, mgd, "f32", "autograd grad_depth")
    _gpu.assert_within(feat.grad.cpu().numpy(), rgf, mgf, "f32", "autograd grad_feat")

"""Every output element at the four largest workloads against the oracle.

The headline (6 views, 40x100, D=118, C=80, fp32), large (4 samples,
40x110, D=118, fp16 in and out, 256x256 grid), train (8 samples, 16x44,
D=118, fp32) and voxel3d (the headline rig into a 128x128x16 voxel grid)
workloads are compared over the whole output (and large's plan once more
with float32 data, whose items are cut at the big size): the forward of
both the interval-table path and the scheduled path, and grad_depth and
grad_feat of both backward paths, each element within
tol * sum|terms| + 1e-6 of the float64 oracle (section 2.1: the
per-voxel sum of depth score times image feature; the gradients by the
chain rule).  Each workload's inputs and oracle results are computed once
per module.  Mass conservation and the adjoint identity are checked as
well, as properties that hold at any size.
"""

import numpy as np
import pytest
import torch

import _gpu
import oracle
from paper_2211_17111_amd import bevpool as bp
from workloads import CONFIGS, draw_inputs, frustum_coor

pytestmark = pytest.mark.gpu

NAMES = ["headline", "large", "train", "voxel3d"]
_CACHE: dict = {}


def _case(name):
    """Inputs, GPU plan and schedule, and oracle forward of a workload."""
    if name not in _CACHE:
        cfg = CONFIGS[name]
        _gpu.say(f"[{name}] inputs and oracle forward")
        coor = frustum_coor(cfg)
        data = draw_inputs(cfg)
        ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, cfg.shape())
        plan = _gpu.run_prepare(coor, cfg.shape())
        sched = bp.schedule(plan)
        _CACHE[name] = dict(cfg=cfg, coor=coor, data=data, ref=ref, mag=mag, plan=plan,
                            sched=sched, dev={k: _gpu.to_dev(v) for k, v in data.items()})
    return _CACHE[name]


def _grads(name):
    c = _case(name)
    if "gref" not in c:
        _gpu.say(f"[{name}] oracle backward")
        c["gref"] = oracle.backward_ref(c["data"]["grad_out"], c["data"]["depth"],
                                        c["data"]["feat"], c["coor"], c["cfg"].shape())
    return c["gref"]


@pytest.fixture(scope="module", autouse=True)
def _drop_cache():
    yield
    _CACHE.clear()


@pytest.mark.parametrize("path", ["ranges", "scheduled"])
@pytest.mark.parametrize("name", NAMES)
def test_forward_every_element(name, path):
    c = _case(name)
    cfg = c["cfg"]
    d, f = c["dev"]["depth"], c["dev"]["feat"]
    odt = _gpu.torch_dtype(cfg.out_dtype)
    _gpu.say(f"[{name}] forward {path}")
    if path == "scheduled":
        out = bp.forward_scheduled(d, f, c["sched"], out_dtype=odt)
    else:
        out = bp.forward(d, f, c["plan"], out_dtype=odt)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    _gpu.assert_within(got, c["ref"], c["mag"], cfg.dtype, f"{name} forward {path}", log=True)
    # empty cells are exactly +0.0
    empty = ~c["mag"].reshape(cfg.cells, cfg.C).any(axis=1)
    rows = got.reshape(cfg.cells, cfg.C)[empty]
    assert np.all(rows == 0.0) and not np.signbit(rows).any()
    # mass conservation per channel (float64 sum of the GPU output)
    kept = oracle.kept_mask(c["coor"], cfg.shape()).reshape(cfg.B, cfg.N, cfg.D, cfg.H, cfg.W)
    dep = c["data"]["depth"].astype(np.float64)
    fea = c["data"]["feat"].astype(np.float64)
    mass = np.einsum("bndhw,bnhwc->c", dep * kept, fea)
    absmass = np.einsum("bndhw,bnhwc->c", np.abs(dep) * kept, np.abs(fea))
    _gpu.assert_within(got.reshape(-1, cfg.C).astype(np.float64).sum(axis=0), mass, absmass,
                       cfg.dtype, f"{name} mass {path}")


@pytest.mark.parametrize("path", ["plan", "scheduled"])
@pytest.mark.parametrize("name", NAMES)
def test_backward_every_element(name, path):
    c = _case(name)
    cfg = c["cfg"]
    rgd, rgf, mgd, mgf = _grads(name)
    g, d, f = c["dev"]["grad_out"], c["dev"]["depth"], c["dev"]["feat"]
    _gpu.say(f"[{name}] backward {path}")
    if path == "scheduled":
        gd, gf = bp.backward_scheduled(g, d, f, c["sched"])
    else:
        gd, gf = bp.backward(g, d, f, c["plan"])
    torch.cuda.synchronize()
    gd = gd.float().cpu().numpy()
    gf = gf.float().cpu().numpy()
    _gpu.assert_within(gd, rgd, mgd, cfg.dtype, f"{name} grad_depth {path}", log=True)
    _gpu.assert_within(gf, rgf, mgf, cfg.dtype, f"{name} grad_feat {path}", log=True)
    # dropped points get exactly +0.0
    kept = oracle.kept_mask(c["coor"], cfg.shape()).reshape(gd.shape)
    assert np.all(gd[~kept] == 0.0) and not np.signbit(gd[~kept]).any()
    # adjoint identity <grad_out, out> = <grad_depth, depth> = <grad_feat, feat>
    g64 = c["data"]["grad_out"].astype(np.float64)
    lhs = float((g64 * c["ref"]).sum())
    r_d = float((gd.astype(np.float64) * c["data"]["depth"].astype(np.float64)).sum())
    r_f = float((gf.astype(np.float64) * c["data"]["feat"].astype(np.float64)).sum())
    scale = float((np.abs(g64) * c["mag"]).sum())
    tol = _gpu.TOL[cfg.dtype] * scale + 1e-6
    assert abs(r_d - lhs) <= tol and abs(r_f - lhs) <= tol, (lhs, r_d, r_f, tol)


def test_big_items_float32():
    """large's plan with float32 inputs and output: 6.45 M kept points, so
    the schedule's items are cut at ITEM_PAIRS_BIG and the forward runs its
    big-item float32 form (no record read-ahead); every output element
    against the oracle."""
    import dataclasses

    import _sched
    cfg = dataclasses.replace(CONFIGS["large"], dtype="f32", out_dtype="f32")
    _gpu.say("[large, float32] inputs and oracle forward")
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg, with_grad=False)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, cfg.shape())
    plan = _gpu.run_prepare(coor, cfg.shape())
    sched = bp.schedule(plan)
    hdr = sched.buffer[:64].view(torch.int32).cpu()
    assert int(hdr[_sched.HDR["item_pairs"]]) == _sched.ITEM_PAIRS_BIG
    out = bp.forward_scheduled(_gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"]), sched)
    torch.cuda.synchronize()
    _gpu.assert_within(out.cpu().numpy(), ref, mag, "f32", label="large float32, big items", log=True)

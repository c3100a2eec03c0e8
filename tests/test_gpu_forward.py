"""GPU forward pooling against the float64 oracle.

Full-output comparison where the oracle runs in seconds; at the large sizes,
sampled cells (longest intervals, random occupied and empty cells, first and
last cell) plus properties that hold at any size.  Tolerance per element:
|gpu - oracle| <= tol * sum|terms| + 1e-6, tol = 1e-5 (fp32 inputs) or 2e-3
(fp16 inputs, fp32 accumulation).
"""

import numpy as np
import pytest
import torch

import _gpu
import _sched
import oracle
from paper_2211_17111_amd import bevpool as bp
from workloads import CONFIGS, draw_inputs, draw_small, frustum_coor, random_coor

pytestmark = pytest.mark.gpu

PATHS = ["ranges", "scheduled"]


@pytest.fixture(params=PATHS)
def path(request):
    return request.param


def _fwd(path, depth_t, feat_t, plan, out_dtype=None, out=None, sched=None):
    if path == "scheduled":
        sched = sched or bp.schedule(plan)
        return bp.forward_scheduled(depth_t, feat_t, sched, out_dtype=out_dtype, out=out)
    return bp.forward(depth_t, feat_t, plan, out_dtype=out_dtype, out=out)


def _run(depth, feat, coor, shape, out_dtype=None, path="ranges"):
    plan = _gpu.run_prepare(coor, shape)
    odt = _gpu.torch_dtype(out_dtype) if out_dtype else None
    out = _fwd(path, _gpu.to_dev(depth), _gpu.to_dev(feat), plan, out_dtype=odt)
    torch.cuda.synchronize()
    return out, plan


@pytest.mark.parametrize("name", ["tiny", "bevdet"])
def test_forward_full(name, path):
    cfg = CONFIGS[name]
    _gpu.say(f"forward full parity: {name} {path}")
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    out, _ = _run(data["depth"], data["feat"], coor, cfg.shape(), path=path)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, cfg.shape())
    _gpu.assert_within(out.cpu().numpy(), ref, mag, cfg.dtype, name)


@pytest.mark.parametrize("C", [1, 3, 16, 17, 64, 80, 260])
@pytest.mark.parametrize("dtype,out_dtype", [("f32", "f32"), ("f16", "f16"), ("f16", "f32")])
def test_forward_random_channels(C, dtype, out_dtype, path):
    shape = dict(B=2, N=2, D=9, H=7, W=13, C=C, X=12, Y=10, Z=2)
    rng = np.random.default_rng(C)
    coor = random_coor(rng, shape, p_out=0.4)
    data = draw_small(rng, shape, dtype=dtype)
    _gpu.say(f"forward random C={C} {dtype}->{out_dtype} {path}")
    out, _ = _run(data["depth"], data["feat"], coor, shape, out_dtype, path=path)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    _gpu.assert_within(out.float().cpu().numpy(), ref, mag, dtype, f"C={C} {dtype}->{out_dtype}")


def test_forward_misaligned_takes_scalar_path(path):
    shape = dict(B=1, N=2, D=6, H=5, W=9, C=8, X=6, Y=6, Z=1)
    rng = np.random.default_rng(1)
    coor = random_coor(rng, shape)
    data = draw_small(rng, shape)
    plan = _gpu.run_prepare(coor, shape)
    # feat and out offset by one element: not 16-byte aligned
    fbuf = torch.empty(data["feat"].size + 1, dtype=torch.float32, device=_gpu.DEV)
    feat = fbuf[1:].view(data["feat"].shape)
    feat.copy_(torch.from_numpy(data["feat"]))
    obuf = torch.empty(1 * 6 * 6 * 8 + 1, dtype=torch.float32, device=_gpu.DEV)
    out = obuf[1:].view(1, 1, 6, 6, 8)
    _fwd(path, _gpu.to_dev(data["depth"]), feat, plan, out=out)
    torch.cuda.synchronize()
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    _gpu.assert_within(out.cpu().numpy(), ref, mag, "f32", "misaligned")


def test_forward_edge_cases(path):
    shape = dict(B=1, N=1, D=8, H=50, W=60, C=80, X=8, Y=8, Z=1)   # P = 24000
    P = 24000
    rng = np.random.default_rng(2)
    data = draw_small(rng, shape)
    cases = {
        "no point in range": np.full((P, 3), -5, dtype=np.int32),
        "one interval of 24000 points": np.tile(np.array([[4, 2, 0]], dtype=np.int32), (P, 1)),
        "first and last cell only": np.where(rng.random((P, 1)) < 0.5,
                                             np.array([[0, 0, 0]]), np.array([[7, 7, 0]])).astype(np.int32),
        "single point": np.concatenate([np.full((P - 1, 3), -1, dtype=np.int32),
                                        np.array([[3, 3, 0]], dtype=np.int32)]),
    }
    for label, coor in cases.items():
        _gpu.say(f"forward edge case: {label} {path}")
        out, _ = _run(data["depth"], data["feat"], coor, shape, path=path)
        ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
        _gpu.assert_within(out.cpu().numpy(), ref, mag, "f32", label)
        occupied = mag.reshape(-1, 80).any(axis=1)
        assert np.all(out.cpu().numpy().reshape(-1, 80)[~occupied] == 0.0), label


@pytest.mark.parametrize("case", ["one cell from many strips", "two cells over many items",
                                  "many small cells", "tall image", "wide fp16 channels",
                                  "wide fp32 channels"])
def test_forward_strip_paths(case, path):
    """Shapes that drive the scheduled kernel through its less common paths:
    a cell summed from many strips' slots, strips cut into several items whose
    segments span many lane groups, strips cut in height, and channel counts
    needing several 64-vector chunks."""
    rng = np.random.default_rng(5)
    dtype = "f32"
    if case == "one cell from many strips":
        shape = dict(B=1, N=1, D=8, H=100, W=60, C=80, X=8, Y=8, Z=1)
        P = 48000
        coor = np.tile(np.array([[4, 2, 0]], dtype=np.int32), (P, 1))
        coor[rng.random(P) < 0.1] = -1       # some points out of range
    elif case == "two cells over many items":
        shape = dict(B=1, N=1, D=40, H=20, W=8, C=8, X=8, Y=8, Z=1)
        P = 40 * 20 * 8
        coor = np.tile(np.array([[4, 2, 0]], dtype=np.int32), (P, 1))
        coor.reshape(40, -1, 3)[1::2, :, 0] = 5   # every point its own pair
    elif case == "many small cells":
        shape = dict(B=1, N=2, D=3, H=30, W=40, C=80, X=64, Y=64, Z=1)
        coor = random_coor(rng, shape, p_out=0.2)
    elif case == "tall image":
        shape = dict(B=2, N=1, D=6, H=150, W=9, C=64, X=16, Y=16, Z=1)
        coor = random_coor(rng, shape, p_out=0.2)
    elif case == "wide fp16 channels":
        shape = dict(B=1, N=2, D=5, H=6, W=7, C=520, X=6, Y=5, Z=1)
        coor = random_coor(rng, shape, p_out=0.2)
        dtype = "f16"
    else:
        shape = dict(B=1, N=2, D=5, H=6, W=7, C=1024, X=6, Y=5, Z=1)
        coor = random_coor(rng, shape, p_out=0.2)
    data = draw_small(rng, shape, dtype=dtype)
    _gpu.say(f"forward strip path: {case} {path}")
    out, _ = _run(data["depth"], data["feat"], coor, shape, path=path)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    _gpu.assert_within(out.float().cpu().numpy(), ref, mag, dtype, case)


def test_forward_nan_free_and_empty_exact_zero(path):
    # Poison the output buffer first: every element must be overwritten.
    cfg = CONFIGS["bevdet"]
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    plan = _gpu.run_prepare(coor, cfg.shape())
    out = torch.full((1, 1, 128, 128, 64), float("nan"), device=_gpu.DEV)
    _fwd(path, _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"]), plan, out=out)
    o = out.cpu().numpy().reshape(-1, 64)
    assert np.isfinite(o).all()
    occ = np.zeros(o.shape[0], dtype=bool)
    occ[plan.ranks_bev.cpu().numpy()] = True
    assert np.all(o[~occ] == 0.0) and np.signbit(o[~occ]).sum() == 0


def _sample_cells(plan, cells, rng, k=120):
    st = plan.interval_starts.cpu().numpy()
    ln = plan.interval_lengths.cpu().numpy()
    rb = plan.ranks_bev.cpu().numpy()
    occ_cells = rb[st]
    longest = occ_cells[np.argsort(ln)[-20:]]
    rand_occ = rng.choice(occ_cells, size=min(k, occ_cells.size), replace=False)
    empty = np.setdiff1d(np.arange(cells), occ_cells)
    rand_empty = rng.choice(empty, size=min(20, empty.size), replace=False) if empty.size else empty
    return np.unique(np.concatenate([longest, rand_occ, rand_empty, [0, cells - 1]]))


@pytest.mark.parametrize("name", ["headline", "large", "train"])
def test_forward_full_size_sampled(name, path):
    cfg = CONFIGS[name]
    _gpu.say(f"forward sampled parity: {name} {path}")
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg, with_grad=False)
    out, plan = _run(data["depth"], data["feat"], coor, cfg.shape(), cfg.out_dtype, path=path)
    rng = np.random.default_rng(7)
    cells = _sample_cells(plan, cfg.cells, rng)
    ref, mag = oracle.forward_cells_ref(data["depth"], data["feat"], coor, cfg.shape(), cells)
    got = out.reshape(cfg.cells, cfg.C)[torch.from_numpy(cells).to(_gpu.DEV)].float().cpu().numpy()
    _gpu.assert_within(got, ref, mag, cfg.dtype, name)
    # mass conservation over the whole output, in float64 on the host
    kept = oracle.kept_mask(coor, cfg.shape()).reshape(cfg.B, cfg.N, cfg.D, cfg.H, cfg.W)
    mass = np.einsum("bndhw,bnhwc->c", data["depth"].astype(np.float64) * kept,
                     data["feat"].astype(np.float64))
    absmass = np.einsum("bndhw,bnhwc->c", np.abs(data["depth"].astype(np.float64)) * kept,
                        np.abs(data["feat"].astype(np.float64)))
    total = out.double().reshape(cfg.cells, cfg.C).sum(dim=0).cpu().numpy()
    _gpu.assert_within(total, mass, absmass, cfg.dtype, f"{name} mass")


def test_forward_deterministic_and_batch_consistent(path):
    cfg = CONFIGS["large"]
    _gpu.say(f"forward determinism + batch consistency: large {path}")
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg, with_grad=False)
    out1, plan = _run(data["depth"], data["feat"], coor, cfg.shape(), "f32", path=path)
    out2 = _fwd(path, _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"]), plan,
                out_dtype=torch.float32)
    assert torch.equal(out1, out2)   # bitwise reproducible run to run
    # Sample 0 of the B=4 run and a B=1 run on sample 0's inputs both match the
    # oracle.  They need not be bitwise equal: the fp32 summation order of a
    # cell depends on where its points fall among the equal work ranges.
    one = dict(cfg.shape(), B=1)
    per = cfg.P // cfg.B
    plan1 = _gpu.run_prepare(coor[:per], one)
    o = _fwd(path, _gpu.to_dev(data["depth"][:1]), _gpu.to_dev(data["feat"][:1]), plan1,
             out_dtype=torch.float32)
    ref, mag = oracle.forward_ref(data["depth"][:1], data["feat"][:1], coor[:per], one)
    _gpu.assert_within(o.cpu().numpy(), ref, mag, "f16", "B=1 run")
    _gpu.assert_within(out1[:1].cpu().numpy(), ref, mag, "f16", "sample 0 of B=4 run")


def test_forward_with_oracle_plan():
    # The plan is plain arrays at the boundary: the oracle's plan drives the GPU.
    cfg = CONFIGS["bevdet"]
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg, with_grad=False)
    ref_plan = oracle.prepare_ref(coor, cfg.shape())
    plan = bp.Plan(cfg.shape(), *(_gpu.to_dev(ref_plan[k]) for k in
                                  ("ranks_depth", "ranks_feat", "ranks_bev",
                                   "interval_starts", "interval_lengths")),
                   ref_plan["n_valid"], ref_plan["n_intervals"])
    out = bp.forward(_gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"]), plan)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, cfg.shape())
    _gpu.assert_within(out.cpu().numpy(), ref, mag, "f32", "oracle plan")


def _check_schedule(coor, shape, label):
    plan = _gpu.run_prepare(coor, shape)
    sched = bp.schedule(plan)
    ref_plan = oracle.prepare_ref(coor, shape)
    got = _sched.decode(sched.buffer.cpu().numpy(), shape, plan.n_valid, plan.n_intervals)
    # items are cut at one share per workgroup of this device's forward
    assert got["n"]["shares"] >= 1, label
    want = _sched.derive(ref_plan, shape, shares=got["n"]["shares"])
    assert got["n"] == want["n"], (label, got["n"], want["n"])
    for k in want:
        if k != "n":
            np.testing.assert_array_equal(got[k], want[k], err_msg=f"{label}: {k}")
    return want


@pytest.mark.parametrize("name", ["tiny", "bevdet", "headline", "large", "train", "voxel3d"])
def test_schedule_matches_numpy(name):
    """Every array of the GPU-built schedule against a numpy derivation from
    the oracle's plan (integer data: bit-exact)."""
    cfg = CONFIGS[name]
    _gpu.say(f"schedule vs numpy: {name}")
    want = _check_schedule(frustum_coor(cfg), cfg.shape(), name)
    if name == "headline":
        # a strip's pairs fall into few cells: far fewer segments than pairs
        assert want["n"]["segs"] < 0.05 * want["n"]["pairs"]


def test_schedule_edge_shapes():
    rng = np.random.default_rng(11)
    shapes = [
        dict(B=2, N=2, D=9, H=7, W=13, C=17, X=12, Y=10, Z=2),   # C not a multiple of 8
        dict(B=1, N=1, D=8, H=100, W=60, C=80, X=8, Y=8, Z=1),   # few cells, many pairs
        dict(B=1, N=2, D=3, H=30, W=40, C=80, X=64, Y=64, Z=1),  # many cells of few pairs
        dict(B=3, N=1, D=4, H=5, W=6, C=16, X=300, Y=7, Z=3),    # X, Y far apart
    ]
    for i, shape in enumerate(shapes):
        _gpu.say(f"schedule edge shape {i}: {shape}")
        _check_schedule(random_coor(rng, shape, p_out=0.3), shape, f"shape {i}")
    shape = shapes[1]
    P = shape["B"] * shape["N"] * shape["D"] * shape["H"] * shape["W"]
    one = np.tile(np.array([[4, 2, 0]], dtype=np.int32), (P, 1))
    want = _check_schedule(one, shape, "one cell")
    assert want["n"]["comb"] == 1 and want["n"]["slots"] == want["n"]["items"]
    shape = dict(B=1, N=1, D=40, H=20, W=8, C=8, X=8, Y=8, Z=1)
    two = np.tile(np.array([[4, 2, 0]], dtype=np.int32), (40 * 20 * 8, 1))
    two.reshape(shape["D"], -1, 3)[1::2, :, 0] = 5   # every point its own pair
    want = _check_schedule(two, shape, "two cells")
    assert want["n"]["items"] > want["n"]["strips"]   # strips cut into several items


@pytest.mark.parametrize("label,shape", [
    # strips of 32 x 3 pixels (C = 80) over D bins: the build by strips in LDS
    # takes up to 12288 points per strip and keys (cell within the sample,
    # pixel, bin) of up to 32 bits; past either bound the general builder runs
    ("12288 points per strip", dict(B=1, N=1, D=128, H=32, W=6, C=80, X=40, Y=40, Z=1)),
    ("12384 points per strip", dict(B=1, N=1, D=129, H=32, W=6, C=80, X=40, Y=40, Z=1)),
    ("32-bit keys", dict(B=1, N=1, D=128, H=32, W=3, C=80, X=512, Y=512, Z=1)),
    ("33-bit keys", dict(B=1, N=1, D=128, H=32, W=3, C=80, X=512, Y=512, Z=2)),
    # 2^21 cells: the cell scans take chunks of 2048 cells (at most 1024 chunks)
    ("2^21 cells", dict(B=1, N=1, D=8, H=32, W=6, C=80, X=1024, Y=1024, Z=2)),
])
def test_schedule_local_bounds(label, shape):
    """Shapes on both sides of the bounds of the strip-local build give the
    schedule of the definitions (both builders are exact)."""
    rng = np.random.default_rng(23)
    _gpu.say(f"schedule at the local-build bounds: {label}")
    _check_schedule(random_coor(rng, shape, p_out=0.3), shape, label)


def test_scheduled_matches_ranges():
    cfg = CONFIGS["headline"]
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg, with_grad=False)
    plan = _gpu.run_prepare(coor, cfg.shape())
    d, f = _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"])
    a = bp.forward(d, f, plan)
    sched = bp.schedule(plan)
    b = bp.forward_scheduled(d, f, sched)
    c = bp.forward_scheduled(d, f, sched)
    assert torch.equal(b, c)
    # both within float32 rounding of each other relative to the output scale
    assert float((a - b).abs().max()) <= 1e-4 * float(a.abs().max())


@pytest.mark.parametrize("name", ["bevdet", "headline"])
def test_scheduled_without_shares(name):
    """A schedule whose items were not cut for this launch's workgroups (here:
    its header says a share is too long) is walked with an equal count of
    each die's items instead; only the balance changes, so the result is the
    same bit for bit."""
    import copy
    cfg = CONFIGS[name]
    _gpu.say(f"forward without shares: {name}")
    data = draw_inputs(cfg, with_grad=False)
    plan = _gpu.run_prepare(frustum_coor(cfg), cfg.shape())
    sched = bp.schedule(plan)
    d, f = _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"])
    want = bp.forward_scheduled(d, f, sched)
    other = copy.copy(sched)
    other.buffer = sched.buffer.clone()
    hdr = other.buffer[:64].view(torch.int32)
    assert int(hdr[_sched.HDR["shares_ok"]]) == 1
    hdr[_sched.HDR["shares_ok"]] = 0
    got = bp.forward_scheduled(d, f, other)
    torch.cuda.synchronize()
    assert torch.equal(got, want)


def test_scheduled_workspace_reuse():
    """One workspace serves a run of forwards over two plans of one shape, with
    new inputs each time: every result equals a fresh workspace's bit for bit
    (the workspace is scratch)."""
    cfg = CONFIGS["bevdet"]
    shape = cfg.shape()
    rng = np.random.default_rng(5)
    plans = [_gpu.run_prepare(c, shape) for c in (frustum_coor(cfg), random_coor(rng, shape, p_out=0.3))]
    scheds = [bp.schedule(p) for p in plans]
    n = max(bp.bevpool_forward_scheduled_workspace_size(shape, s.n_slots) for s in scheds)
    ws = torch.full((n,), 0xFF, dtype=torch.uint8, device=_gpu.DEV)  # NaN rows before the first use
    for t in range(4):
        _gpu.say(f"workspace reuse: forward {t}")
        data = draw_inputs(cfg, seed=100 + t, with_grad=False)
        d, f = _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"])
        s = scheds[t % 2]
        fresh = bp.forward_scheduled(d, f, s)
        reused = bp.forward_scheduled(d, f, s, workspace=ws)
        torch.cuda.synchronize()
        assert s.n_slots > 0
        assert torch.equal(fresh, reused), t


def test_scheduled_workspace_checked():
    """A workspace smaller than the schedule's slot count needs is refused
    with BEVPOOL_EWORKSPACE before anything is enqueued: `out` keeps its
    contents."""
    cfg = CONFIGS["bevdet"]
    shape = cfg.shape()
    data = draw_inputs(cfg, with_grad=False)
    plan = _gpu.run_prepare(frustum_coor(cfg), shape)
    sched = bp.schedule(plan)
    d, f = _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"])
    n = bp.bevpool_forward_scheduled_workspace_size(shape, sched.n_slots)
    assert n > 0
    small = torch.zeros(n - 4, dtype=torch.uint8, device=_gpu.DEV)
    out = torch.full((cfg.B, cfg.Z, cfg.Y, cfg.X, cfg.C), 7.0, device=_gpu.DEV)
    with pytest.raises(bp.BevpoolError) as err:
        bp.forward_scheduled(d, f, sched, out=out, workspace=small)
    assert err.value.status == bp.BEVPOOL_EWORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


@pytest.mark.parametrize("case", ["slots", "unbuilt", "item size"])
def test_scheduled_header_mismatch_nan(case):
    """A schedule whose header does not hold the counts of the call (another
    slot count, a buffer no build has written, or items cut at the other
    size) gives NaN in every element of `out`, never a partial or stale
    result."""
    cfg = CONFIGS["bevdet"]
    shape = cfg.shape()
    data = draw_inputs(cfg, with_grad=False)
    plan = _gpu.run_prepare(frustum_coor(cfg), shape)
    sched = bp.schedule(plan)
    d, f = _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"])
    n_slots = sched.n_slots
    buf = sched.buffer
    if case == "slots":
        n_slots += 1
    elif case == "item size":
        # a schedule cut at the other item size than this launch's rule gives
        buf = sched.buffer.clone()
        hdr = buf[:64].view(torch.int32)
        want = _sched.item_pairs(plan.n_valid)
        assert int(hdr[_sched.HDR["item_pairs"]]) == want
        hdr[_sched.HDR["item_pairs"]] = _sched.ITEM_PAIRS_BIG + _sched.ITEM_PAIRS - want
    else:
        buf = torch.zeros_like(sched.buffer)
    ws = torch.empty(bp.bevpool_forward_scheduled_workspace_size(shape, n_slots) + 16, dtype=torch.uint8,
                     device=_gpu.DEV)
    out = torch.zeros((cfg.B, cfg.Z, cfg.Y, cfg.X, cfg.C), device=_gpu.DEV)
    code = bp.BEVPOOL_F32
    bp.bevpool_forward_scheduled(shape, code, code, d, f, buf, buf.numel(), plan.n_valid, plan.n_intervals,
                                 n_slots, out, ws, ws.numel())
    torch.cuda.synchronize()
    assert bool(torch.isnan(out).all())



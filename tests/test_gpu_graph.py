"""Graph capture of the whole path.

prepare, schedule, the scheduled forward and the scheduled backward make no
memset, copy, synchronisation or allocation call (every buffer, workspaces
included, is the caller's), so a caller can capture them in one HIP graph.
The graph is replayed several times, with eager work and synchronisations
between the replays, and every replay must give the eager results bit for
bit (integer plan and schedule, and the floating-point outputs, whose
summation order the schedule fixes).
"""

import pytest
import torch

import _gpu
from paper_2211_17111_amd import bevpool as bp
from workloads import CONFIGS, draw_inputs, frustum_coor

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    cfg = CONFIGS["bevdet"]
    shape = cfg.shape()
    _gpu.say("graph capture: prepare + schedule + forward + backward (bevdet)")
    data = draw_inputs(cfg)
    coor = _gpu.to_dev(frustum_coor(cfg))
    depth, feat, grad_out = (_gpu.to_dev(data[k]) for k in ("depth", "feat", "grad_out"))
    plan = bp.prepare(coor, shape)
    nv, ni = plan.n_valid, plan.n_intervals
    dev = depth.device
    P = cfg.P
    i32 = dict(dtype=torch.int32, device=dev)
    rd, rf, rb = (torch.empty(P, **i32) for _ in range(3))
    cap = min(P, cfg.cells)
    st, ln, cnt = torch.empty(cap, **i32), torch.empty(cap, **i32), torch.empty(2, **i32)
    ws_p = torch.empty(bp.bevpool_prepare_workspace_size(shape), dtype=torch.uint8, device=dev)
    sb, wb = bp.bevpool_schedule_size(shape, nv, ni)
    sched = torch.empty(sb, dtype=torch.uint8, device=dev)
    ws_s = torch.empty(wb, dtype=torch.uint8, device=dev)
    n_slots = bp.schedule(plan).n_slots  # (the header, read back once before capture)
    fb = bp.bevpool_forward_scheduled_workspace_size(shape, n_slots)
    ws_f = torch.empty(max(fb, 16), dtype=torch.uint8, device=dev)
    out = torch.empty((cfg.B, cfg.Z, cfg.Y, cfg.X, cfg.C), dtype=torch.float32, device=dev)
    gd, gf = torch.empty_like(depth), torch.empty_like(feat)
    code = bp.BEVPOOL_F32

    def run():  # everything on the current stream
        bp.bevpool_prepare(shape, coor, rd, rf, rb, st, ln, cnt, ws_p, ws_p.numel())
        bp.bevpool_schedule(shape, rd, rb, nv, ni, sched, sb, ws_s, ws_s.numel())
        bp.bevpool_forward_scheduled(shape, code, code, depth, feat, sched, sb, nv, ni, n_slots, out,
                                     ws_f, fb)
        bp.bevpool_backward_scheduled(shape, code, code, grad_out, depth, feat, sched, sb, nv, ni, gd, gf)

    # (the plan and schedule arrays are written only up to their counts: every
    # output is cleared before the eager run as before each replay, so that
    # the regions nothing writes compare equal)
    outputs = (rd, rf, rb, st, ln, cnt, sched, out, gd, gf)
    for t in outputs:
        t.zero_()
    run()
    torch.cuda.synchronize()
    want = [t.clone() for t in outputs]
    assert [int(x) for x in cnt.cpu()] == [nv, ni]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()  # (a warm-up on the capture's stream, as torch asks)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    for k in range(3):
        for t in outputs:  # eager work between replays: clear every output again
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, got, ref in zip(("rd", "rf", "rb", "starts", "lengths", "counts", "schedule", "out",
                                   "grad_depth", "grad_feat"), outputs, want):
            assert torch.equal(got, ref), (k, name)

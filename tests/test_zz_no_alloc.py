"""The allocation-free scheduled forward (bevpool_forward_scheduled_noalloc).

Called through the C ABI, it must give exactly what
bevpool_forward_scheduled gives with a workspace (the same kernels, with the
slots in the library's static device array instead): two calls in a row,
the second with a smaller input, each compared element by element.
"""

import pytest
import torch

import _gpu
from paper_2211_17111_amd import bevpool as bp
from workloads import CONFIGS, draw_inputs, frustum_coor

pytestmark = pytest.mark.gpu

_DT = {"f32": torch.float32, "f16": torch.float16}


def _compare(name):
    cfg = CONFIGS[name]
    shape = cfg.shape()
    _gpu.say(f"allocation-free forward vs workspace forward: {name}")
    data = draw_inputs(cfg, with_grad=False)
    plan = _gpu.run_prepare(frustum_coor(cfg), shape)
    sched = bp.schedule(plan)
    assert bp.bevpool_forward_scheduled_workspace_size(shape, sched.n_slots) <= bp.NOALLOC_SCRATCH_BYTES
    d, f = _gpu.to_dev(data["depth"]), _gpu.to_dev(data["feat"])
    odt = _DT[cfg.out_dtype]
    want = bp.forward_scheduled(d, f, sched, out_dtype=odt)
    got = torch.full_like(want, float("nan"))
    bp.bevpool_forward_scheduled_noalloc(shape, bp._DTYPE_CODE[d.dtype], bp._DTYPE_CODE[odt], d, f,
                                         sched.buffer, sched.buffer.numel(), plan.n_valid, plan.n_intervals,
                                         sched.n_slots, got)
    torch.cuda.synchronize()
    assert torch.equal(got, want), name


def test_noalloc_matches_workspace_forward():
    _compare("headline")
    _compare("bevdet")  # (a smaller input after a larger one: the array keeps stale slots)

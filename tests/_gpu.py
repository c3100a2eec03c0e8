"""Helpers shared by the GPU tests: upload, run through the C ABI, compare."""

from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2211_17111_amd import bevpool as bp

DEV = "cuda:0"
TOL = {"f32": 1e-5, "f16": 2e-3}   # relative to the sum of |terms|
ABS = 1e-6


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_prepare(coor: np.ndarray, shape: dict) -> bp.Plan:
    return bp.prepare(to_dev(coor.astype(np.int32)), shape)


def plan_to_numpy(plan: bp.Plan) -> dict:
    return {
        "ranks_depth": plan.ranks_depth.cpu().numpy(),
        "ranks_feat": plan.ranks_feat.cpu().numpy(),
        "ranks_bev": plan.ranks_bev.cpu().numpy(),
        "interval_starts": plan.interval_starts.cpu().numpy(),
        "interval_lengths": plan.interval_lengths.cpu().numpy(),
        "n_valid": plan.n_valid,
        "n_intervals": plan.n_intervals,
    }


def assert_plan_equal(got: dict, ref: dict, label: str = ""):
    assert got["n_valid"] == ref["n_valid"], f"{label} n_valid {got['n_valid']} != {ref['n_valid']}"
    assert got["n_intervals"] == ref["n_intervals"], \
        f"{label} n_intervals {got['n_intervals']} != {ref['n_intervals']}"
    for k in ("ranks_depth", "ranks_feat", "ranks_bev", "interval_starts", "interval_lengths"):
        g, r = got[k], ref[k]
        if not np.array_equal(g, r):
            bad = np.flatnonzero(g != r)
            raise AssertionError(f"{label} {k}: {bad.size} mismatches, first at {bad[0]}: "
                                 f"gpu {g[bad[0]]} vs oracle {r[bad[0]]}")


def assert_within(gpu, ref, mag, dtype: str, label: str = "", log: bool = False) -> float:
    """Every element within tol * sum|terms| + 1e-6 of the oracle; returns the
    worst ratio err / bound (printed when ``log``)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    mag = np.asarray(mag, dtype=np.float64)
    assert gpu.shape == ref.shape, f"{label} shape {gpu.shape} != {ref.shape}"
    err = np.abs(gpu - ref)
    bound = TOL[dtype] * mag + ABS
    bad = ~(err <= bound)
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(bad, err / bound, 0)), err.shape)
        raise AssertionError(f"{label}: {int(bad.sum())} elements out of tolerance; worst at {i}: "
                             f"gpu {gpu[i]} oracle {ref[i]} |terms| {mag[i]}")
    worst = float((err / bound).max()) if err.size else 0.0
    if log:
        say(f"{label}: {err.size} elements within tolerance, worst err/bound {worst:.3e}")
    return worst


def torch_dtype(name: str):
    return {"f32": torch.float32, "f16": torch.float16}[name]

"""Plant plausible mistakes in the CPU oracle and check that a pin catches each.

Every mutant below swaps one oracle helper for a subtly wrong version (a
dropped bound, a transposed rank, an unstable sort, a sign error, a gradient
that leaks into dropped points).  The pins of ``_pins.py`` must reject all of
them, which shows they are sharp enough to trust the unmutated oracle.  All
of this runs on the CPU.
"""

import numpy as np
import pytest

import _pins
import oracle
import oracle.bevpool_ref as ref
from workloads import random_coor, draw_small

SHAPE = dict(B=2, N=2, D=4, H=3, W=3, C=3, X=4, Y=4, Z=2)


def _inputs(seed=21):
    rng = np.random.default_rng(seed)
    coor = random_coor(rng, SHAPE)
    data = draw_small(rng, SHAPE)
    return coor, data


def _all_fails(coor, data):
    checks = [
        lambda: _pins.check_prepare_brute(ref.prepare_ref, coor, SHAPE),
        lambda: _pins.check_prepare_invariants(ref.prepare_ref, coor, SHAPE),
        lambda: _pins.check_forward_brute(ref.forward_ref, data["depth"], data["feat"], coor, SHAPE),
        lambda: _pins.check_forward_identities(ref.forward_ref, data["depth"], data["feat"], coor, SHAPE),
        lambda: _pins.check_backward_brute(ref.backward_ref, data["grad_out"], data["depth"],
                                           data["feat"], coor, SHAPE),
        lambda: _pins.check_backward_identities(ref.backward_ref, ref.forward_ref, data["grad_out"],
                                                data["depth"], data["feat"], coor, SHAPE, n_fd=4),
    ]
    fails = []
    for check in checks:
        try:
            fails += check()
        except Exception as exc:  # a crash on a mutant also counts as caught
            fails.append(f"raised {type(exc).__name__}: {exc}")
    return fails


def test_unmutated_oracle_passes_every_pin():
    coor, data = _inputs()
    assert _all_fails(coor, data) == []


_orig_kept = ref.kept_mask
_orig_ranks = ref.point_ranks
_orig_frustum = ref.frustum_feature


def _kept_inclusive_upper(coor, shape):
    X, Y, Z = shape["X"], shape["Y"], shape["Z"]
    x, y, z = (coor[:, i].astype(np.int64) for i in range(3))
    return (x >= 0) & (x <= X) & (y >= 0) & (y < Y) & (z >= 0) & (z < Z)


def _kept_no_z(coor, shape):
    X, Y = shape["X"], shape["Y"]
    x, y = (coor[:, i].astype(np.int64) for i in range(2))
    return (x >= 0) & (x < X) & (y >= 0) & (y < Y)


def _ranks_feat_hw_swapped(p, coor_p, shape):
    rd, rf, rb = _orig_ranks(p, coor_p, shape)
    H, W = shape["H"], shape["W"]
    w = p % W
    h = (p // W) % H
    bn = p // (W * H * shape["D"])
    return rd, (bn * W + w) * H + h, rb


def _ranks_bev_xy_swapped(p, coor_p, shape):
    rd, rf, rb = _orig_ranks(p, coor_p, shape)
    X, Y, Z, N = shape["X"], shape["Y"], shape["Z"], shape["N"]
    b = p // (shape["W"] * shape["H"] * shape["D"] * N)
    x, y, z = (coor_p[:, i].astype(np.int64) for i in range(3))
    return rd, rf, ((b * Z + z) * X + x) * Y + y


def _ranks_bev_no_batch(p, coor_p, shape):
    rd, rf, rb = _orig_ranks(p, coor_p, shape)
    X, Y = shape["X"], shape["Y"]
    x, y, z = (coor_p[:, i].astype(np.int64) for i in range(3))
    return rd, rf, (z * Y + y) * X + x


def _frustum_sign(depth, feat, b, n):
    return -_orig_frustum(depth, feat, b, n)


def _frustum_feat_of_next_view(depth, feat, b, n):
    n2 = (n + 1) % feat.shape[1]
    dep = depth[b, n].astype(np.float64)
    img = feat[b, n2].astype(np.float64)
    return dep[:, :, :, None] * img[None]


def _unstable_prepare(coor, shape):
    kept = ref.kept_mask(coor, shape)
    p = np.flatnonzero(kept)
    rd, rf, rb = ref.point_ranks(p, coor[p], shape)
    # descending frustum index among ties instead of ascending
    order = np.lexsort((-rd, rb))
    rd, rf, rb = rd[order], rf[order], rb[order]
    _, starts, lengths = np.unique(rb, return_index=True, return_counts=True)
    return {"ranks_depth": rd, "ranks_feat": rf, "ranks_bev": rb,
            "interval_starts": starts, "interval_lengths": lengths,
            "n_valid": int(p.size), "n_intervals": int(starts.size)}


MUTANTS = {
    "upper bound inclusive": ("kept_mask", _kept_inclusive_upper),
    "z bound ignored": ("kept_mask", _kept_no_z),
    "feature rank h/w transposed": ("point_ranks", _ranks_feat_hw_swapped),
    "BEV rank x/y transposed": ("point_ranks", _ranks_bev_xy_swapped),
    "BEV rank drops the sample": ("point_ranks", _ranks_bev_no_batch),
    "frustum feature sign flipped": ("frustum_feature", _frustum_sign),
    "frustum feature from the wrong view": ("frustum_feature", _frustum_feat_of_next_view),
    "ties sorted in descending frustum index": ("prepare_ref", _unstable_prepare),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(ref, attr, fn)
    coor, data = _inputs()
    assert _all_fails(coor, data) != [], f"mutant '{name}' passed every pin"


def test_gradient_leak_is_caught(monkeypatch):
    orig = ref.backward_ref

    def leaky(grad_out, depth, feat, coor, shape):
        gd, gf, gdm, gfm = orig(grad_out, depth, feat, coor, shape)
        kept = _orig_kept(coor, shape).reshape(gd.shape)
        return gd + np.where(kept, 0.0, 1e-3), gf, gdm, gfm

    monkeypatch.setattr(ref, "backward_ref", leaky)
    coor, data = _inputs()
    assert _all_fails(coor, data) != []


def test_transposed_gradient_operand_is_caught(monkeypatch):
    orig = ref.backward_ref

    def wrong(grad_out, depth, feat, coor, shape):
        # grad_feat built from the depth score of the mirrored depth bin
        return orig(grad_out, depth[:, :, ::-1], feat, coor, shape)

    monkeypatch.setattr(ref, "backward_ref", wrong)
    coor, data = _inputs()
    assert _all_fails(coor, data) != []

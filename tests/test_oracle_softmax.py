"""Pins of the oracle's depth softmax (CPU only).

The fused forward takes depth logits: a pixel's depth scores are the softmax
of its logits over the D depth bins (section 2.1 reads the depth score as a
per-pixel distribution over depth classes), and the pooled result is the
ordinary forward on those scores.  The pins fix the log-sum-exp against a
pure-Python evaluation, the softmax's defining properties (positive, sums
to one per pixel over the depth axis only, invariant to a per-pixel shift),
its closed forms (uniform logits give 1/D, a dominant logit a one-hot
score) and the reduction to forward_ref.
"""

import math

import numpy as np
import pytest

import oracle
from workloads import CONFIGS, draw_inputs, frustum_coor, random_coor

SMALL = dict(B=2, N=2, D=5, H=3, W=4, C=3, X=6, Y=5, Z=2)


def _logits(rng, shape, scale=3.0):
    return scale * rng.standard_normal((shape["B"], shape["N"], shape["D"], shape["H"], shape["W"]))


def test_lse_matches_pure_python():
    rng = np.random.default_rng(11)
    x = _logits(rng, SMALL)
    got = oracle.depth_lse_ref(x)
    B, N, D, H, W = x.shape
    for b in range(B):
        for n in range(N):
            for h in range(H):
                for w in range(W):
                    want = math.log(math.fsum(math.exp(float(x[b, n, d, h, w])) for d in range(D)))
                    assert abs(got[b, n, h, w] - want) <= 1e-13 * max(1.0, abs(want))


def test_softmax_is_a_distribution_over_depth():
    rng = np.random.default_rng(12)
    for scale in (3.0, 80.0):  # (80: terms far outside exp's range without the max shift)
        p = oracle.depth_softmax_ref(_logits(rng, SMALL, scale))
        assert np.all(np.isfinite(p)) and np.all(p >= 0)
        assert np.allclose(p.sum(axis=2), 1.0, rtol=0, atol=1e-12)


def test_softmax_shift_invariant_per_pixel():
    """Adding one constant to all logits of a pixel changes nothing; a
    softmax over any other axis would change."""
    rng = np.random.default_rng(13)
    x = _logits(rng, SMALL)
    c = 10.0 * rng.standard_normal((x.shape[0], x.shape[1], 1, x.shape[3], x.shape[4]))
    assert np.allclose(oracle.depth_softmax_ref(x + c), oracle.depth_softmax_ref(x), rtol=1e-12, atol=1e-15)


def test_softmax_closed_forms():
    x = np.zeros((1, 2, 7, 2, 3))
    assert np.allclose(oracle.depth_softmax_ref(x), 1.0 / 7, rtol=1e-15, atol=0)
    y = np.zeros((1, 1, 4, 1, 2))
    y[0, 0, 2, 0, 0] = 1000.0  # dominant: exp(-1000) underflows to exactly 0
    y[0, 0, 0, 0, 1] = 1000.0
    p = oracle.depth_softmax_ref(y)
    assert p[0, 0, :, 0, 0].tolist() == [0.0, 0.0, 1.0, 0.0]
    assert p[0, 0, :, 0, 1].tolist() == [1.0, 0.0, 0.0, 0.0]


def test_forward_softmax_reduces_to_forward_ref():
    rng = np.random.default_rng(14)
    coor = random_coor(rng, SMALL, p_out=0.2)
    x = _logits(rng, SMALL)
    feat = rng.standard_normal((SMALL["B"], SMALL["N"], SMALL["H"], SMALL["W"], SMALL["C"]))
    got, mag = oracle.forward_softmax_ref(x, feat, coor, SMALL)
    depth = np.exp(x - oracle.depth_lse_ref(x)[:, :, None])
    want, want_mag = oracle.forward_ref(depth, feat, coor, SMALL)
    assert np.array_equal(got, want) and np.array_equal(mag, want_mag)
    # uniform logits: every score 1/D
    u, _ = oracle.forward_softmax_ref(np.zeros_like(x), feat, coor, SMALL)
    w, _ = oracle.forward_ref(np.full_like(x, 1.0 / SMALL["D"]), feat, coor, SMALL)
    assert np.allclose(u, w, rtol=1e-14, atol=1e-15)


def test_workload_logits_give_the_workload_scores():
    """draw_inputs' scores are the float64 softmax of the logits it returns
    (rounded to the working precision), so the fused forward of the logits
    is the ordinary forward of the scores to within that rounding."""
    cfg = CONFIGS["tiny"]
    d = draw_inputs(cfg, with_logits=True)
    p = oracle.depth_softmax_ref(d["logits"])
    assert np.allclose(p, d["depth"], rtol=1e-6, atol=1e-7)
    coor = frustum_coor(cfg)
    a, mag = oracle.forward_softmax_ref(d["logits"], d["feat"], coor, cfg.shape())
    b, _ = oracle.forward_ref(d["depth"], d["feat"], coor, cfg.shape())
    assert np.all(np.abs(a - b) <= 1e-5 * mag + 1e-6)


def test_wrong_axis_mutant_caught():
    """A planted mistake (softmax over the width axis) breaks the per-pixel
    normalisation the pins check."""
    rng = np.random.default_rng(15)
    x = _logits(rng, SMALL)
    m = x.max(axis=4, keepdims=True)
    bad = np.exp(x - m) / np.exp(x - m).sum(axis=4, keepdims=True)
    assert not np.allclose(bad.sum(axis=2), 1.0, atol=1e-6)

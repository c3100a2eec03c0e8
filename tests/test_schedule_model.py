"""The block schedule's definitions, executed on the CPU (no GPU).

tests/_blocks.py derives the block schedule from the oracle's plan with numpy
and executes it the way the scheduled forward does: dense weights from the
depth runs of each piece's records, per-block sums of weights times feature
rows, per-cell sums of column partials, then the slots of cells reached from
several strips.  The result must equal the oracle's forward (section 2.1) to
float64 rounding.  This pins the schedule's semantics (a wrong entry, record,
block row range, partial-row index or slot order fails here) before the GPU
build is compared with it bit for bit.
"""

import numpy as np
import pytest

import _blocks
import oracle
from workloads import CONFIGS, draw_inputs, draw_small, frustum_coor, random_coor


def _check(coor, shape, data, label):
    plan = oracle.prepare_ref(coor, shape)
    sch = _blocks.derive(plan, shape)
    got = _blocks.execute(sch, data["depth"], data["feat"])
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    err = np.abs(got - ref)
    assert np.all(err <= 1e-12 * mag + 1e-300), f"{label}: max err {err.max():.3e}"
    return plan, sch


@pytest.mark.parametrize("name", ["tiny", "bevdet"])
def test_schedule_executes_to_oracle(name):
    cfg = CONFIGS[name]
    _check(frustum_coor(cfg), cfg.shape(), draw_inputs(cfg), name)


@pytest.mark.parametrize("seed", range(4))
def test_schedule_random_shapes(seed):
    rng = np.random.default_rng(100 + seed)
    shapes = [dict(B=2, N=2, D=9, H=7, W=13, C=5, X=12, Y=10, Z=2),
              dict(B=1, N=3, D=17, H=5, W=9, C=3, X=6, Y=6, Z=1),
              dict(B=3, N=1, D=4, H=5, W=6, C=4, X=300, Y=7, Z=3),
              dict(B=1, N=1, D=40, H=20, W=8, C=2, X=8, Y=8, Z=1)]
    shape = shapes[seed]
    coor = random_coor(rng, shape, p_out=0.3)
    _check(coor, shape, draw_small(rng, shape), f"shape {seed}")


def test_schedule_edge_cases():
    shape = dict(B=1, N=1, D=8, H=50, W=60, C=3, X=8, Y=8, Z=1)
    P = 8 * 50 * 60
    rng = np.random.default_rng(2)
    data = draw_small(rng, shape)
    one = np.tile(np.array([[4, 2, 0]], dtype=np.int32), (P, 1))
    plan, sch = _check(one, shape, data, "one cell")
    # one TC per strip, one slot per strip, one combined cell
    assert sch["header"][_blocks.HDR["comb"]] == 1
    assert sch["header"][_blocks.HDR["slots"]] == sch["header"][_blocks.HDR["tcs"]] == 15
    single = np.full((P, 3), -1, dtype=np.int32)
    single[1234] = [3, 3, 0]
    _check(single, shape, data, "single point")
    two = one.copy()
    two.reshape(8, -1, 3)[1::2, :, 0] = 5   # every point its own pair
    _, sch = _check(two, shape, data, "alternating cells")
    assert sch["header"][_blocks.HDR["pairs"]] == P


def test_schedule_invariants():
    """Structural facts the kernels rely on (headline rig, bevdet shape)."""
    cfg = CONFIGS["bevdet"]
    shape = cfg.shape()
    plan = oracle.prepare_ref(frustum_coor(cfg), shape)
    s = _blocks.derive(plan, shape)
    h = s["header"]
    K, SW = _blocks.K, _blocks.SW
    npairs = int(h[_blocks.HDR["pairs"]])
    # every kept point lies in exactly one pair
    assert int(s["pair_n"].sum()) == plan["n_valid"]
    # pieces partition blocks, TCs, CCs and records in order
    pc = s["piece"]
    for col, ncol in ((5, 6), (7, 8), (9, 10), (11, 12)):
        assert pc[0, col] == 0 and np.all(pc[1:, col] == pc[:-1, col] + pc[:-1, ncol])
    assert pc[-1, 7] + pc[-1, 8] == npairs
    assert np.all(pc[:, 10] <= _blocks.tc_max(shape["H"]))
    assert np.all(pc[:, 13] <= _blocks.ENT_BUDGET) and np.all(pc[:, 12] <= 256)
    # records address entries inside their piece's weight array
    for j in range(len(pc)):
        strip, plo, nh, dlo, nd, blk0, nblk, rec0, nrec, tc0, ntc, cc0, ncc, nent, pix0, ncol = pc[j]
        recs = s["rec"][rec0:rec0 + nrec]
        assert np.all((recs & 0x7FF) + ((recs >> 11) & 0x1FFF) < nd)
        assert np.all((recs >> 24) < ncc)
        cct = s["cc"][cc0:cc0 + ncc]
        assert np.all((cct & 0xFFFF) < nent)
        blocks = s["block"][blk0:blk0 + nblk]
        assert np.all(blocks[:, 3] + K * blocks[:, 2] <= nent)
        assert np.all(((blocks[:, 0] >> 8) & 0xFF) <= K)
        prs = s["tc"][tc0:tc0 + ntc, 1]
        for c in range(SW):
            pr = (prs >> (8 * c)) & 0xFF
            assert np.all((pr == 0xFF) | (pr < nblk * K))
    # slots: the comb table lists each shared cell's slots contiguously
    slots = int(h[_blocks.HDR["slots"]])
    assert s["comb_slot0"][0] == 0 and s["comb_slot0"][-1] == slots
    assert np.all(np.diff(s["comb_slot0"]) >= 2)
    dest = s["tc"][:, 0]
    assert np.array_equal(np.sort(~dest[dest < 0]), np.arange(slots))


def test_schedule_mutant_caught():
    """A planted mistake in how entries are addressed (row stride K - 1)
    makes the executed schedule disagree with the oracle."""
    cfg = CONFIGS["tiny"]
    shape = cfg.shape()
    coor = frustum_coor(cfg)
    data = draw_inputs(cfg)
    plan = oracle.prepare_ref(coor, shape)
    sch = _blocks.derive(plan, shape)
    saved = _blocks.K
    try:
        _blocks.K = saved - 1
        got = _blocks.execute(sch, data["depth"], data["feat"])
    except (IndexError, ValueError):
        return  # an out-of-range entry is caught too
    finally:
        _blocks.K = saved
    ref, _ = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    assert not np.allclose(got, ref)

"""The strip schedule's definitions, executed on the CPU (no GPU).

tests/_sched.py derives the schedule from the oracle's plan with numpy; here a
plain interpreter walks that schedule the way the scheduled forward does
(strip rows addressed from the strip number, pair weights from depth runs,
segments cut by head bits, direct stores versus slots, then the slot
combination and the empty-cell fill) and the result must equal the oracle's
forward (section 2.1) to float64 rounding.  This pins the schedule's
semantics (a wrong strip geometry, pair run, segment cut or slot order fails
here) before any GPU compares its buffers against it bit for bit.
"""

import numpy as np
import pytest

import _sched
import oracle
from workloads import CONFIGS, draw_inputs, draw_small, frustum_coor, random_coor


def _execute(sch, depth, feat, shape):
    """Forward from a derived schedule, in float64; also counts the stores of
    every output row."""
    B, N, D, H, W, C = (shape[k] for k in "BNDHWC")
    cells = B * shape["Z"] * shape["Y"] * shape["X"]
    hw = H * W
    sd = _sched.strip_dims(shape)
    dflat = depth.reshape(-1).astype(np.float64)
    fflat = feat.reshape(-1, C).astype(np.float64)
    out = np.full((cells, C), np.nan)
    writes = np.zeros(cells, dtype=np.int64)
    slots = np.full((sch["n"]["slots"], C), np.nan)
    per = sd["nhb"] * sd["nwb"]
    for i in range(sch["n"]["items"]):
        s = int(sch["item_strip"][i])
        bn, r = divmod(s, per)
        hb, wb = divmod(r, sd["nwb"])
        h0, w0 = hb * sd["bh"], wb * sd["bw"]
        bws = min(sd["bw"], W - w0)
        npix = min(sd["bh"], H - h0) * bws
        rows = [(bn * H + h0 + lp // bws) * W + w0 + lp % bws for lp in range(npix)]
        p0, p1 = sch["item_pair0"][i], sch["item_pair0"][i + 1]
        g0, g1 = sch["item_seg0"][i], sch["item_seg0"][i + 1]
        assert 1 <= p1 - p0 <= sch["n"]["item_pairs"]
        seg = -1
        acc = {}
        for k in range(p0, p1):
            ln = int(sch["pair_ln"][k])
            if ln & _sched.PAIR_HEAD:
                seg += 1
            assert k > p0 or ln & _sched.PAIR_HEAD
            assert sch["pair_seg"][k] == seg
            lp, n = ln & (_sched.PAIR_HEAD - 1), ln >> 16
            assert lp < npix and n >= 1
            rd0 = int(sch["pair_rd0"][k])
            w = sum(dflat[rd0 + j * hw] for j in range(n))
            acc[seg] = acc.get(seg, 0.0) + w * fflat[rows[lp]]
        assert seg + 1 == g1 - g0
        for j, v in acc.items():
            dest = int(sch["seg_dest"][g0 + j])
            if dest >= 0:
                out[dest] = v
                writes[dest] += 1
            else:
                assert np.isnan(slots[~dest]).all()
                slots[~dest] = v
    for j, cell in enumerate(sch["comb_cell"]):
        a, b = sch["comb_slot0"][j], sch["comb_slot0"][j + 1]
        assert b - a >= 2
        out[cell] = slots[a:b].sum(axis=0)
        writes[cell] += 1
    out[sch["empty"]] = 0.0
    writes[sch["empty"]] += 1
    return out, writes


def _check(depth, feat, coor, shape, label, shares=1):
    plan = oracle.prepare_ref(coor, shape)
    sch = _sched.derive(plan, shape, shares=shares)
    out, writes = _execute(sch, depth, feat, shape)
    assert (writes == 1).all(), f"{label}: rows written {np.bincount(writes)} times"
    ref, mag = oracle.forward_ref(depth, feat, coor, shape)
    ref = ref.reshape(out.shape)
    mag = mag.reshape(out.shape)
    assert np.all(np.abs(out - ref) <= 1e-12 * mag + 1e-300), label
    return sch


@pytest.mark.parametrize("shares", [1, 256])
def test_schedule_model_tiny(shares):
    cfg = CONFIGS["tiny"]
    data = draw_inputs(cfg, with_grad=False)
    sch = _check(data["depth"], data["feat"], frustum_coor(cfg), cfg.shape(), "tiny", shares)
    assert sch["n"]["slots"] == 0 or sch["n"]["comb"] > 0


@pytest.mark.parametrize("shares", [1, 256])
def test_schedule_model_bevdet_geometry(shares):
    cfg = CONFIGS["bevdet"]
    data = draw_inputs(cfg, with_grad=False)
    sch = _check(data["depth"], data["feat"], frustum_coor(cfg), cfg.shape(), "bevdet", shares)
    # pixel columns see few cells: far fewer segments than pairs
    assert sch["n"]["segs"] < 0.25 * sch["n"]["pairs"]


@pytest.mark.parametrize("shape", [
    dict(B=2, N=2, D=9, H=7, W=13, C=17, X=12, Y=10, Z=2),
    dict(B=1, N=1, D=8, H=100, W=60, C=80, X=8, Y=8, Z=1),    # strips cut in height
    dict(B=1, N=2, D=3, H=30, W=40, C=300, X=64, Y=64, Z=1),  # one-pixel-wide strips
    dict(B=3, N=1, D=4, H=5, W=6, C=16, X=300, Y=7, Z=3),
])
@pytest.mark.parametrize("shares", [1, 8, 1000])
def test_schedule_model_random(shape, shares):
    rng = np.random.default_rng(shape["C"])
    data = draw_small(rng, shape)
    _check(data["depth"], data["feat"], random_coor(rng, shape, p_out=0.3), shape, str(shape), shares)


@pytest.mark.parametrize("shares", [1, 3, 8, 64, 5000])
def test_shares_cut_items(shares):
    # every share boundary starts an item, so share w's items hold exactly its
    # pairs [floor(P w / S), floor(P (w + 1) / S)); items stay inside one strip
    # and hold at most the schedule's item size in pairs
    cfg = CONFIGS["bevdet"]
    plan = oracle.prepare_ref(frustum_coor(cfg), cfg.shape())
    sch = _sched.derive(plan, cfg.shape(), shares=shares)
    P = sch["n"]["pairs"]
    ip0 = sch["item_pair0"]
    si = sch["share_item0"]
    assert si.size == shares + 1 and si[0] == 0 and si[-1] == sch["n"]["items"]
    s_p0 = np.r_[ip0[:-1][np.r_[True, sch["item_strip"][1:] != sch["item_strip"][:-1]]], P]
    def bound(w):  # floor(P w / S), moved to a strip end closer than MIN_PIECE
        c = (P * w) // shares
        if 0 < c < P:
            j = np.searchsorted(s_p0, c, side="right") - 1
            a, b = s_p0[j], s_p0[j + 1]
            c = a if c - a < _sched.MIN_PIECE else (b if b - c < _sched.MIN_PIECE else c)
        return c
    for w in range(shares):
        lo, hi = bound(w), bound(w + 1)
        assert lo <= hi
        if lo < hi:
            assert ip0[si[w]] == lo and ip0[si[w + 1]] == hi
        else:
            assert si[w] == si[w + 1]
        assert hi - lo <= P // shares + 1 + 2 * _sched.MIN_PIECE
    # a share cut inside a strip leaves at least MIN_PIECE pairs on each side
    for w in range(1, shares):
        c = bound(w)
        j = np.searchsorted(s_p0, c, side="right") - 1
        assert c == s_p0[j] or min(c - s_p0[j], s_p0[j + 1] - c) >= _sched.MIN_PIECE
    assert np.all(np.diff(ip0) >= 1) and np.all(np.diff(ip0) <= sch["n"]["item_pairs"])
    # every strip starts an item
    strip_p0 = ip0[:-1][np.r_[True, sch["item_strip"][1:] != sch["item_strip"][:-1]]]
    base = _sched.derive(plan, cfg.shape(), shares=1)
    assert np.array_equal(strip_p0, base["item_pair0"][:-1][np.r_[True, base["item_strip"][1:] !=
                                                                   base["item_strip"][:-1]]])
    assert sch["n"]["shares_ok"] == int(np.diff(si).max() <= _sched.SHARE_ITEMS)


def test_schedule_model_one_cell():
    # every point in one cell: strips of many pairs are cut into several items,
    # so the cell has one slot per item
    shape = dict(B=1, N=1, D=40, H=20, W=8, C=8, X=8, Y=8, Z=1)
    rng = np.random.default_rng(5)
    data = draw_small(rng, shape)
    P = shape["D"] * shape["H"] * shape["W"]
    coor = np.tile(np.array([[4, 2, 0]], dtype=np.int32), (P, 1))
    # alternate two cells along depth so that every point is its own pair
    coor.reshape(shape["D"], -1, 3)[1::2, :, 0] = 5
    sch = _check(data["depth"], data["feat"], coor, shape, "one cell")
    assert sch["n"]["items"] > sch["n"]["strips"]
    assert sch["n"]["comb"] == 2


def test_strip_dims_budget():
    # a strip's rows of one 64-vector channel chunk fit the LDS budget
    for C in (1, 16, 64, 80, 256, 300, 4096):
        sd = _sched.strip_dims(dict(B=1, N=1, H=40, W=100, C=C))
        assert sd["pixels"] * 4 * min(C, 256) <= _sched.STRIP_BYTES or sd["pixels"] == 1
    sd = _sched.strip_dims(dict(B=1, N=6, H=40, W=100, C=80))
    assert (sd["bh"], sd["bw"], sd["strips"]) == (40, 2, 300)


def _walk_partition(sch, depth, feat, shape, G):
    """The scheduled forward's in-item work split, executed on the CPU: an
    item's pairs are cut into G equal ranges; a range sums its segments,
    stores the ones it holds whole, keeps the part of a segment it starts
    inside (handed to the range holding that segment's start) and of one it
    ends inside (which then adds the following ranges' parts in order)."""
    B, N, D, H, W, C = (shape[k] for k in "BNDHWC")
    hw = H * W
    cells = B * shape["Z"] * shape["Y"] * shape["X"]
    sd = _sched.strip_dims(shape)
    dflat = depth.reshape(-1).astype(np.float64)
    fflat = feat.reshape(-1, C).astype(np.float64)
    out = np.full((cells, C), np.nan)
    slots = np.full((sch["n"]["slots"], C), np.nan)
    per = sd["nhb"] * sd["nwb"]

    def store(dest, v):
        target = out[dest] if dest >= 0 else slots[~dest]
        assert np.isnan(target).all()
        target[:] = v

    for i in range(sch["n"]["items"]):
        s = int(sch["item_strip"][i])
        bn, r = divmod(s, per)
        hb, wb = divmod(r, sd["nwb"])
        h0, w0 = hb * sd["bh"], wb * sd["bw"]
        bws = min(sd["bw"], W - w0)
        p0, p1 = sch["item_pair0"][i], sch["item_pair0"][i + 1]
        np_ = p1 - p0
        g0 = sch["item_seg0"][i]
        ln = sch["pair_ln"][p0:p1]
        head = (ln & _sched.PAIR_HEAD) != 0
        seg = sch["pair_seg"][p0:p1]
        lp = ln & (_sched.PAIR_HEAD - 1)
        n = ln >> 16
        rd0 = sch["pair_rd0"][p0:p1]
        rows = (bn * H + h0 + lp // bws) * W + w0 + lp % bws
        wts = np.array([sum(dflat[rd0[k] + j * hw] for j in range(n[k])) for k in range(np_)])
        dest = sch["seg_dest"][g0:]
        rb = lambda g: (g * np_) // G
        first, last = {}, {}
        for g in range(G):
            kb, ke = rb(g), rb(g + 1)
            if kb >= ke:
                continue
            prev_cont = not head[kb]
            next_cont = ke < np_ and not head[ke]
            cur, pend, acc = seg[kb], prev_cont, np.zeros(C)
            for k in range(kb, ke):
                if head[k] and k != kb:
                    if pend:
                        first[g], pend = acc, False
                    else:
                        store(dest[cur], acc)
                    acc, cur = np.zeros(C), cur + 1
                acc = acc + wts[k] * fflat[rows[k]]
            if pend:
                first[g] = acc
            elif next_cont:
                last[g] = (acc, seg[ke - 1])
            else:
                store(dest[cur], acc)
        for g, (v, sg) in last.items():
            total = v.copy()
            for g2 in range(g + 1, G):
                b2, e2 = rb(g2), rb(g2 + 1)
                if b2 >= e2:
                    continue
                if head[b2]:
                    break
                total += first[g2]
                if not (seg[e2 - 1] == sg and e2 < np_ and not head[e2]):
                    break
            store(dest[sg], total)
    for j, c in enumerate(sch["comb_cell"]):
        out[c] = slots[sch["comb_slot0"][j]:sch["comb_slot0"][j + 1]].sum(axis=0)
    out[sch["empty"]] = 0.0
    return out


@pytest.mark.parametrize("G", [1, 7, 36, 64, 5000])
def test_walk_partition_model(G):
    # every output row written once and equal to the oracle, whatever the
    # number of ranges (more ranges than pairs included)
    shape = dict(B=1, N=2, D=12, H=6, W=5, C=8, X=6, Y=6, Z=1)
    rng = np.random.default_rng(G)
    data = draw_small(rng, shape)
    coor = random_coor(rng, shape, p_out=0.2)
    coor[::3, 0] = coor[0, 0]  # long segments across ranges
    plan = oracle.prepare_ref(coor, shape)
    sch = _sched.derive(plan, shape)
    out = _walk_partition(sch, data["depth"], data["feat"], shape, G)
    ref, mag = oracle.forward_ref(data["depth"], data["feat"], coor, shape)
    ref = ref.reshape(out.shape)
    assert np.all(np.abs(out - ref) <= 1e-12 * mag.reshape(out.shape) + 1e-300)


def test_item_size_rule(monkeypatch):
    """Items are big (ITEM_PAIRS_BIG) from BIG_ITEM_POINTS kept points on,
    else ITEM_PAIRS; a schedule's items respect its size, and big items are
    used where pieces are long enough (the threshold lowered here so that
    bevdet's plan takes both sizes)."""
    assert _sched.item_pairs(_sched.BIG_ITEM_POINTS) == _sched.ITEM_PAIRS_BIG
    assert _sched.item_pairs(_sched.BIG_ITEM_POINTS - 1) == _sched.ITEM_PAIRS
    cfg = CONFIGS["bevdet"]
    plan = oracle.prepare_ref(frustum_coor(cfg), cfg.shape())
    n_valid = int(plan["n_valid"])
    for limit, want in ((n_valid, _sched.ITEM_PAIRS_BIG), (n_valid + 1, _sched.ITEM_PAIRS)):
        monkeypatch.setattr(_sched, "BIG_ITEM_POINTS", limit)
        sch = _sched.derive(plan, cfg.shape(), shares=1)
        assert sch["n"]["item_pairs"] == want
        sizes = np.diff(sch["item_pair0"])
        assert sizes.min() >= 1 and sizes.max() <= want
        if want == _sched.ITEM_PAIRS_BIG:
            assert sizes.max() > _sched.ITEM_PAIRS

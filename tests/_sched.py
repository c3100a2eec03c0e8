"""Host-side reading of a schedule and a numpy derivation of it.

The schedule (see paper_2211_17111_amd/csrc/internal.h) is integer data built
on the GPU from a plan; these helpers decode the device buffer and derive the
same arrays independently with numpy from the oracle's plan, so the GPU
schedule can be checked bit for bit.
"""

from __future__ import annotations

import numpy as np

ALIGN = 256
ITEM_PAIRS = 2048
ITEM_PAIRS_BIG = 3072      # items of a schedule whose shares hold many kept points
BIG_ITEM_POINTS = 16384 * 256    # kept points from which items are big
STRIP_BYTES = 32 * 1024
PAIR_HEAD = 1 << 15
MAX_SHARES = 1024
SHARE_ITEMS = 128
MIN_PIECE = 512
HDR = dict(pairs=0, items=1, segs=2, valid=3, occ=4, occ_found=5, empty=6, slots=7, comb=8, strips=9,
           shares=10, shares_ok=11, item_pairs=12)


def item_pairs(n_valid: int) -> int:
    """The item size a schedule of n_valid kept points is cut at."""
    return ITEM_PAIRS_BIG if n_valid >= BIG_ITEM_POINTS else ITEM_PAIRS


def strip_dims(shape) -> dict:
    C, H, W = shape["C"], shape["H"], shape["W"]
    R = max(1, STRIP_BYTES // (4 * min(C, 256)))
    bh = min(H, R)
    bw = max(1, min(W, R // bh))
    nhb, nwb = -(-H // bh), -(-W // bw)
    return dict(bh=bh, bw=bw, nhb=nhb, nwb=nwb, strips=shape["B"] * shape["N"] * nhb * nwb,
                pixels=bh * bw)


def layout(shape, n_valid: int, n_occ: int) -> dict:
    cells = shape["B"] * shape["Z"] * shape["Y"] * shape["X"]
    sd = strip_dims(shape)
    nv = max(n_valid, 1)
    nocc = n_occ + 1
    n_empty = max(cells - n_occ, 0)
    icap = sd["strips"] + n_valid // ITEM_PAIRS + MAX_SHARES + 2
    rows = shape["B"] * shape["N"] * shape["H"] * shape["W"]
    sizes = [("header", 16), ("pair_rd0", nv), ("pair_ln", nv), ("pair_seg", (nv + 1) // 2),
             ("item_strip", icap),
             ("item_pair0", icap + 1), ("item_seg0", icap + 1), ("seg_dest", nv),
             ("comb_cell", nocc), ("comb_slot0", nocc), ("empty", n_empty + 1),
             ("bp_cell", nv), ("bp_dn", nv), ("pix_pair0", rows + 1),
             ("share_item0", MAX_SHARES + 1)]
    off, out = 0, {}
    for name, n in sizes:
        out[name] = (off // 4, n)
        off += -(-4 * n // ALIGN) * ALIGN
    out["total"] = off
    return out


def decode(buf: np.ndarray, shape, n_valid: int, n_occ: int) -> dict:
    """Arrays of a schedule buffer (bytes) with their valid lengths."""
    ints = buf.view(np.int32)
    lay = layout(shape, n_valid, n_occ)
    lay.pop("total")
    arr = {k: ints[o:o + n].copy() for k, (o, n) in lay.items()}
    h = arr["header"]
    n = {k: int(h[i]) for k, i in HDR.items()}
    np_, ni, ns, nc = n["pairs"], n["items"], n["segs"], n["comb"]
    return dict(
        n=n,
        pair_rd0=arr["pair_rd0"][:np_].astype(np.int64),
        pair_ln=arr["pair_ln"][:np_].view(np.uint32).astype(np.int64),
        pair_seg=arr["pair_seg"].view(np.uint16)[:np_].astype(np.int64),
        item_strip=arr["item_strip"][:ni].astype(np.int64),
        item_pair0=arr["item_pair0"][:ni + 1].astype(np.int64),
        item_seg0=arr["item_seg0"][:ni + 1].astype(np.int64),
        seg_dest=arr["seg_dest"][:ns].astype(np.int64),
        comb_cell=arr["comb_cell"][:nc].astype(np.int64),
        comb_slot0=arr["comb_slot0"][:nc + 1].astype(np.int64),
        empty=arr["empty"][:n["empty"]].astype(np.int64),
        bp_cell=arr["bp_cell"][:np_].astype(np.int64),
        bp_dn=arr["bp_dn"][:np_].view(np.uint32).astype(np.int64),
        pix_pair0=arr["pix_pair0"].astype(np.int64),
        share_item0=arr["share_item0"][:n["shares"] + 1].astype(np.int64) if n["shares"] > 0
        else np.zeros(0, dtype=np.int64),
    )


def snap(c: int, a: int, b: int) -> int:
    """A share boundary c inside strip [a, b), moved to a strip end closer
    than MIN_PIECE pairs."""
    return a if c - a < MIN_PIECE else (b if b - c < MIN_PIECE else c)


def strip_items(a: int, b: int, P: int, S: int, ip: int = ITEM_PAIRS) -> list:
    """First pairs of the items of a strip with pairs [a, b): cut at the
    (snapped) share boundaries floor(P w / S) inside it, each piece of L pairs
    into ceil(L / ip) items at floor(i L / K) of the piece."""
    raw = [c for c in ((P * w) // S for w in range(1, S)) if a < c < b]
    cuts = sorted({snap(c, a, b) for c in raw} - {a, b})
    starts = []
    for q, e in zip([a] + cuts, cuts + [b]):
        L = e - q
        K = -(-L // ip)
        starts += [q + (i * L) // K for i in range(K)]
    return starts


def derive(plan: dict, shape, shares: int = 1) -> dict:
    """The schedule of a plan, by the definitions, in numpy; items cut at
    `shares` equal shares of the pairs."""
    rd = plan["ranks_depth"].astype(np.int64)
    rb = plan["ranks_bev"].astype(np.int64)
    H, W, D = shape["H"], shape["W"], shape["D"]
    hw, per_view = H * W, D * H * W
    cells = shape["B"] * shape["Z"] * shape["Y"] * shape["X"]
    sd = strip_dims(shape)
    bh, bw, nhb, nwb = sd["bh"], sd["bw"], sd["nhb"], sd["nwb"]
    row = (rd // per_view) * hw + rd % hw
    bn, h, w = row // hw, (row % hw) // W, row % W
    strip = (bn * nhb + h // bh) * nwb + w // bw
    w0 = (w // bw) * bw
    lp = (h % bh) * np.minimum(bw, W - w0) + (w - w0)
    o = np.lexsort((np.arange(rd.size), lp, rb, strip))
    rd, rb, row, strip, lp = rd[o], rb[o], row[o], strip[o], lp[o]
    n = rd.size
    head = np.ones(n, dtype=bool)
    head[1:] = (rb[1:] != rb[:-1]) | (row[1:] != row[:-1]) | (rd[1:] != rd[:-1] + hw)
    hp = np.flatnonzero(head)
    npts = np.diff(np.r_[hp, n])
    p_rb, p_row, p_strip, p_lp, p_rd0 = rb[hp], row[hp], strip[hp], lp[hp], rd[hp]
    p_d0 = (p_rd0 % per_view) // hw
    npairs = hp.size
    # items: strips cut at the shares, pieces cut into at most ip pairs
    ip = item_pairs(n)
    s_head = np.r_[True, p_strip[1:] != p_strip[:-1]]
    s_p0 = np.r_[np.flatnonzero(s_head), npairs]
    item_strip, item_pair0 = [], []
    for j in range(s_p0.size - 1):
        st = strip_items(int(s_p0[j]), int(s_p0[j + 1]), int(npairs), shares, ip)
        item_strip += [int(p_strip[s_p0[j]])] * len(st)
        item_pair0 += st
    item_start = np.zeros(npairs, dtype=bool)
    item_start[item_pair0] = True
    seg_head = item_start.copy()
    seg_head[1:] |= p_rb[1:] != p_rb[:-1]
    seg_head[0] = True
    seg_p0 = np.flatnonzero(seg_head)
    seg_cell = p_rb[seg_p0]
    nsegs = seg_p0.size
    item_seg0 = np.searchsorted(seg_p0, item_pair0)
    pair_ln = p_lp | np.where(seg_head, PAIR_HEAD, 0) | (npts << 16)
    pair_item = np.searchsorted(np.array(item_pair0), np.arange(npairs), side="right") - 1
    pair_seg = (np.cumsum(seg_head) - 1) - item_seg0[pair_item]
    # slots: segments sorted by cell (stably); cells with several segments
    so = np.argsort(seg_cell, kind="stable")
    keys = seg_cell[so]
    shared = np.zeros(nsegs, dtype=bool)
    shared[1:] |= keys[1:] == keys[:-1]
    shared[:-1] |= keys[:-1] == keys[1:]
    slot = np.cumsum(shared) - shared
    seg_dest = np.empty(nsegs, dtype=np.int64)
    seg_dest[so] = np.where(shared, ~slot, keys)
    run_head = np.r_[True, keys[1:] != keys[:-1]]
    comb = run_head & shared
    comb_cell = keys[comb]
    comb_slot0 = np.r_[slot[comb], int(shared.sum())]
    occ = np.zeros(cells, dtype=bool)
    occ[keys] = True
    empty = np.flatnonzero(~occ)
    # pixel-major pairs: stable by feature row
    po = np.argsort(p_row, kind="stable")
    bp_cell, bp_dn = p_rb[po], (p_d0 | (npts << 16))[po]
    n_rows = shape["B"] * shape["N"] * H * W
    pix_pair0 = np.searchsorted(p_row[po], np.arange(n_rows + 1), side="left")
    n_items = len(item_pair0)
    def bound(w):
        c = (npairs * w) // shares
        if 0 < c < npairs:
            j = int(np.searchsorted(s_p0, c, side="right")) - 1
            c = snap(c, int(s_p0[j]), int(s_p0[j + 1]))
        return c
    bounds = [bound(w) for w in range(shares + 1)]
    share_item0 = np.searchsorted(np.array(item_pair0, dtype=np.int64), bounds, side="left")
    shares_ok = int(np.diff(share_item0).max() <= SHARE_ITEMS)
    return dict(
        n=dict(pairs=int(npairs), items=n_items, segs=int(nsegs), valid=n, occ=int(run_head.sum()),
               occ_found=int(run_head.sum()), empty=int(empty.size), slots=int(shared.sum()),
               comb=int(comb.sum()), strips=int(s_p0.size - 1), shares=shares, shares_ok=shares_ok,
               item_pairs=ip),
        pair_rd0=p_rd0, pair_ln=pair_ln, pair_seg=pair_seg, item_strip=np.array(item_strip, dtype=np.int64),
        item_pair0=np.r_[np.array(item_pair0, dtype=np.int64), npairs],
        item_seg0=np.r_[item_seg0, nsegs].astype(np.int64), seg_dest=seg_dest,
        comb_cell=comb_cell, comb_slot0=comb_slot0, empty=empty,
        bp_cell=bp_cell, bp_dn=bp_dn, pix_pair0=pix_pair0, share_item0=share_item0.astype(np.int64))

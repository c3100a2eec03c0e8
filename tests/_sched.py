"""Host-side reading of a forward schedule and a numpy derivation of it.

The schedule (see paper_2211_17111_amd/csrc/internal.h) is integer data built
on the GPU from a plan; these helpers decode the device buffer and derive the
same arrays independently with numpy from the oracle's plan, so the GPU
schedule can be checked bit for bit.
"""

from __future__ import annotations

import numpy as np

ALIGN = 256
TILE_PAIRS = 4096
TILE_THREADS = 1024
TILE_MAX_CELLS = 512
TILE_ITEM_BYTES = 192 * 1024
XCDS = 8
HDR = dict(pairs=0, tiles=1, items=2, valid=3, occ=4, occ_found=5, empty=6, row_entries=7, work=8)


def _bit_length(v: int) -> int:
    b = 1
    while (1 << b) < v:
        b += 1
    return b


def slice_counts(C: int) -> list[int]:
    ks = [k for k in range(1, C + 1) if C % k == 0 and (k == 1 or (C // k) % 8 == 0)]
    return ks[:16]


def max_units(vec: int) -> int:
    return 8 if vec == 1 else 16 // vec


def groups(cs: int, vec: int) -> int:
    g = min(64, -(-cs // vec))
    return (TILE_THREADS // 64) * (64 // g)


def max_cells(C: int) -> int:
    best = TILE_MAX_CELLS
    for vec in (1, 4, 8):
        if C % vec:
            continue
        best = min(best, (max_units(vec) - 1) * groups(min(C, 64 * vec), vec))
    return max(best, 1)


def morton_level(shape) -> int:
    L = 0
    while (1 << L) < shape["X"] or (1 << L) < shape["Y"]:
        L += 1
    if L > 15 or _bit_length(shape["B"] * shape["Z"]) + 2 * L > 31:
        return -1
    return L


def _spread(v):
    v = v.astype(np.uint64) & 0xFFFF
    out = np.zeros_like(v)
    for b in range(16):
        out |= ((v >> b) & 1) << (2 * b)
    return out


def cell_key(rb, shape):
    L = morton_level(shape)
    rb = rb.astype(np.int64)
    if L < 0:
        return rb
    XY = shape["X"] * shape["Y"]
    bz, r = rb // XY, rb % XY
    y, x = r // shape["X"], r % shape["X"]
    return (bz << (2 * L)) | (_spread(x) | (_spread(y) << 1)).astype(np.int64)


def layout(shape, n_valid: int, n_occ: int) -> dict:
    cells = shape["B"] * shape["Z"] * shape["Y"] * shape["X"]
    nv = max(n_valid, 1)
    nocc = n_occ + 1
    n_empty = max(cells - n_occ, 0)
    items_cap = (n_occ + 1) * slice_counts(shape["C"])[-1]
    rows = shape["B"] * shape["N"] * shape["H"] * shape["W"]
    sizes = [("header", 16), ("pair_rl", nv), ("pair_dn", nv), ("cell_out", nocc),
             ("cell_pair", nocc), ("tile_cell", nocc), ("tile_row0", nocc), ("rows", nv),
             ("row_dbase", nv), ("empty", n_empty + 1), ("bp_cell", nv), ("bp_dn", nv),
             ("pix_pair0", rows + 1), ("item_tile", items_cap), ("item_slice", items_cap),
             ("xcd_begin", XCDS + 1)]
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
    np_ = n["pairs"]
    nt = n["tiles"]
    return dict(
        n=n,
        pair_rl=arr["pair_rl"][:np_].astype(np.int64),
        pair_dn=arr["pair_dn"][:np_].view(np.uint32).astype(np.int64),
        cell_out=arr["cell_out"][:n_occ].astype(np.int64),
        cell_pair=arr["cell_pair"][:n_occ + 1].astype(np.int64),
        tile_cell=arr["tile_cell"][:nt + 1].astype(np.int64),
        tile_row0=arr["tile_row0"][:nt + 1].astype(np.int64),
        rows=arr["rows"][:n["row_entries"]].astype(np.int64),
        row_dbase=arr["row_dbase"][:n["row_entries"]].astype(np.int64),
        empty=arr["empty"][:n["empty"]].astype(np.int64),
        bp_cell=arr["bp_cell"][:np_].astype(np.int64),
        bp_dn=arr["bp_dn"][:np_].view(np.uint32).astype(np.int64),
        pix_pair0=arr["pix_pair0"].astype(np.int64),
        item_tile=arr["item_tile"][:n["items"]].astype(np.int64),
        item_slice=arr["item_slice"][:n["items"]].astype(np.int64),
        xcd_begin=arr["xcd_begin"].astype(np.int64),
    )


def derive(plan: dict, shape) -> dict:
    """The schedule of a plan, by the definitions, in numpy."""
    rd = plan["ranks_depth"].astype(np.int64)
    rb = plan["ranks_bev"].astype(np.int64)
    H, W, D, C = shape["H"], shape["W"], shape["D"], shape["C"]
    hw, per_view = H * W, D * H * W
    cells = shape["B"] * shape["Z"] * shape["Y"] * shape["X"]
    row = (rd // per_view) * hw + rd % hw
    key = cell_key(rb, shape)
    o = np.lexsort((np.arange(rd.size), row, key))
    rd, rb, row, key = rd[o], rb[o], row[o], key[o]
    n = rd.size
    head = np.ones(n, dtype=bool)
    head[1:] = (rb[1:] != rb[:-1]) | (row[1:] != row[:-1]) | (rd[1:] != rd[:-1] + hw)
    hp = np.flatnonzero(head)
    npts = np.diff(np.r_[hp, n])
    p_rb, p_row = rb[hp], row[hp]
    p_d0 = (rd[hp] % per_view) // hw
    cell_head = np.ones(hp.size, dtype=bool)
    cell_head[1:] = p_rb[1:] != p_rb[:-1]
    cell_pair = np.r_[np.flatnonzero(cell_head), hp.size]
    cell_out = p_rb[cell_head]
    n_occ = cell_out.size
    # tiles
    T = TILE_PAIRS // 2
    cmax = max_cells(C)
    cnt = np.diff(cell_pair)
    big = cnt > T
    c = np.arange(n_occ)
    th = (c % cmax == 0)
    th[1:] |= big[1:] | big[:-1] | (cell_pair[1:-1] // T != cell_pair[:-2] // T)
    tile_cell = np.r_[np.flatnonzero(th), n_occ]
    cell_tile = np.cumsum(th) - 1
    pair_tile = np.repeat(cell_tile, cnt)
    # distinct rows per tile
    tr = np.unique(np.stack([pair_tile, p_row], 1), axis=0)
    tile_row0 = np.r_[np.searchsorted(tr[:, 0], np.arange(tile_cell.size - 1)), len(tr)]
    rows = tr[:, 1]
    row_dbase = (rows // hw) * per_view + rows % hw
    entry = np.searchsorted(tr[:, 0] * (1 << 32) + tr[:, 1], pair_tile * (1 << 32) + p_row)
    pair_rl = entry - tile_row0[pair_tile]
    pair_dn = p_d0 | (npts << 16)
    # pixel-major pairs: stable by feature row (cell-key order kept within a pixel)
    po = np.argsort(p_row, kind="stable")
    bp_cell, bp_dn = p_rb[po], pair_dn[po]
    n_rows = shape["B"] * shape["N"] * H * W
    pix_pair0 = np.searchsorted(p_row[po], np.arange(n_rows + 1), side="left")
    occ = np.zeros(cells, dtype=bool)
    occ[cell_out] = True
    empty = np.flatnonzero(~occ)
    # items
    ks = slice_counts(C)
    n_rows_t = np.diff(tile_row0)
    n_pairs_t = cell_pair[tile_cell[1:]] - cell_pair[tile_cell[:-1]]
    item_tile, item_slice, work = [], [], []
    for t in range(tile_cell.size - 1):
        K = next((k for k in ks if n_rows_t[t] * (C // k) * 4 <= TILE_ITEM_BYTES), ks[-1])
        w = min(((n_rows_t[t] + n_pairs_t[t] // 2) * (C // K) + 63) // 64, 0x3FFFFFFF)
        for k in range(K):
            item_tile.append(t)
            item_slice.append(k | (K << 16))
            work.append(w)
    work = np.array(work, dtype=np.int64)
    cum = np.cumsum(work)
    total = int(cum[-1]) if cum.size else 0
    n_items = len(item_tile)
    xcd = [0] * (XCDS + 1)
    xcd[XCDS] = n_items
    for x in range(1, XCDS):
        b = (total * x + XCDS - 1) // XCDS
        idx = np.flatnonzero(cum >= b)
        xcd[x] = int(idx[0]) + 1 if idx.size else n_items   # first item preceded by >= b
    return dict(
        n=dict(pairs=int(hp.size), tiles=int(tile_cell.size - 1), items=n_items, valid=n,
               occ=n_occ, occ_found=n_occ, empty=int(empty.size), row_entries=int(rows.size),
               work=total),
        pair_rl=pair_rl, pair_dn=pair_dn, cell_out=cell_out, cell_pair=cell_pair,
        tile_cell=tile_cell, tile_row0=tile_row0, rows=rows, row_dbase=row_dbase, empty=empty,
        bp_cell=bp_cell, bp_dn=bp_dn, pix_pair0=pix_pair0,
        item_tile=np.array(item_tile, dtype=np.int64), item_slice=np.array(item_slice, dtype=np.int64),
        xcd_begin=np.array(xcd, dtype=np.int64))

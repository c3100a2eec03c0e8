"""Numpy derivation of the block schedule, and a float64 executor of it.

The block schedule (built on the GPU by bevpool_schedule; layout in
paper_2211_17111_amd/csrc/internal.h) regroups the sorted plan of section
2.1 for the scheduled forward.  ``derive`` computes every array of it from a
plan with plain numpy, following the same integer rules, so the GPU build can
be compared bit for bit; ``pack`` lays the arrays out as the device buffer;
``execute`` runs the forward the way the kernels use the schedule (dense
weights from depth runs, per-block sums, per-piece and cross-strip
combination) in float64, which must equal the oracle's forward.

Terms (all counts are of kept points of the plan):
  strip   SW adjacent feature-map columns of one (sample, camera) image, all
          H rows
  pair    a maximal run of one pixel's kept points in one cell over
          consecutive depth bins (first bin d0, n points)
  TC      (strip, cell) with at least one pair; within a strip TCs are
          ordered by (least d0, cell)
  piece   a run of consecutive TCs of one strip: a new piece starts at the
          strip's first TC, at every TCMAX-th TC and where the strip's pair
          count before the TC crosses a multiple of PAIRS.  One piece is one
          workgroup of the forward.
  CC      (TC, column of the strip) with at least one pair; within a piece,
          CCs are ordered by (column, least d0, cell)
  block   K consecutive CCs of one column of a piece: the dense weight
          matrix of its CCs over the column's rows [hlo, hlo + nu), stored
          row-major as entry ebase + u * K + k within the piece
"""

from __future__ import annotations

import numpy as np

SW = 4             # strip width (columns)
K = 12             # cells per block
PAIRS = 3000       # pairs per piece (cut where the running count crosses a multiple)
ENT_BUDGET = 8192  # weight entries a piece may need at most
HDR_WORDS = 16
PIECE_WORDS = 16
BLOCK_WORDS = 4
ALIGN = 256

HDR = dict(pairs=0, pieces=1, blocks=2, valid=3, occ=4, occ_found=5, empty=6, slots=7, comb=8,
           tcs=9, ccs=10, max_ent=11, max_blk=12, max_pix=13, pixrec=14, max_rec=15)
PIECE = dict(strip=0, plo=1, nh=2, dlo=3, nd=4, blk0=5, nblk=6, rec0=7, nrec=8, tc0=9, ntc=10,
             cc0=11, ncc=12, nent=13, pix0=14, ncol=15)


def tc_max(H: int) -> int:
    """TCs per piece: blocks of a piece times K times H stay within ENT_BUDGET."""
    return K * max(0, min(4, ENT_BUDGET // (SW * K * H)))


def derive(plan: dict, shape: dict) -> dict:
    B, N, D, H, W = (int(shape[k]) for k in "BNDHW")
    X, Y, Z = (int(shape[k]) for k in "XYZ")
    cells = B * Z * Y * X
    HW = H * W
    nsw = -(-W // SW)
    tcmax = tc_max(H)
    assert tcmax > 0 and D <= 2048
    nv = int(plan["n_valid"])
    rd = plan["ranks_depth"][:nv].astype(np.int64)
    rb = plan["ranks_bev"][:nv].astype(np.int64)
    w = rd % W
    h = (rd // W) % H
    d = (rd // HW) % D
    bn = rd // (D * HW)
    strip = bn * nsw + w // SW
    wl = w % SW
    lp_strip = h * SW + wl                         # pixel within the strip

    # pairs: points ordered by (strip, cell, pixel, plan position); a pair
    # starts where any of them changes or the depth bin is not the next one
    order = np.lexsort((np.arange(nv), lp_strip, rb, strip))
    so, co, po, do = strip[order], rb[order], lp_strip[order], d[order]
    head = np.ones(nv, dtype=bool)
    head[1:] = (so[1:] != so[:-1]) | (co[1:] != co[:-1]) | (po[1:] != po[:-1]) | (do[1:] != do[:-1] + 1)
    ph = np.flatnonzero(head)
    npairs = ph.size
    p_n = np.diff(np.r_[ph, nv])
    p_strip, p_cell, p_lp, p_d0 = so[ph], co[ph], po[ph], do[ph]
    p_h, p_wl = p_lp // SW, p_lp % SW
    p_rd0 = rd[order][ph]

    # TCs: runs of equal (strip, cell) over the pairs
    th = np.ones(npairs, dtype=bool)
    th[1:] = (p_strip[1:] != p_strip[:-1]) | (p_cell[1:] != p_cell[:-1])
    tc_p0 = np.flatnonzero(th)
    ntc = tc_p0.size
    tc_of_pair = np.cumsum(th) - 1
    tc_strip, tc_cell = p_strip[tc_p0], p_cell[tc_p0]
    tc_pairs = np.diff(np.r_[tc_p0, npairs])
    tc_dmin = np.minimum.reduceat(p_d0, tc_p0)
    # TC order: (strip, dmin, cell); TCs are in (strip, cell) order already
    tord = np.lexsort((np.arange(ntc), tc_dmin, tc_strip))
    rank_of_tc = np.empty(ntc, np.int64)
    rank_of_tc[tord] = np.arange(ntc)
    s_sorted = tc_strip[tord]
    sstart = np.r_[True, s_sorted[1:] != s_sorted[:-1]]
    first_rank = np.maximum.accumulate(np.where(sstart, np.arange(ntc), 0))
    r_in = np.arange(ntc) - first_rank
    cum_excl = np.cumsum(tc_pairs[tord]) - tc_pairs[tord]
    cum_in = cum_excl - cum_excl[first_rank]
    prev_cum_in = np.r_[-1, cum_in[:-1]]
    bnd = sstart | (r_in % tcmax == 0) | (cum_in // PAIRS != prev_cum_in // PAIRS)
    piece_of_rank = np.cumsum(bnd) - 1
    npc = int(piece_of_rank[-1]) + 1 if ntc else 0
    pc_rank0 = np.flatnonzero(bnd)                 # first TC rank of each piece
    pc_ntc = np.diff(np.r_[pc_rank0, ntc])
    pc_strip = s_sorted[pc_rank0]
    piece_of_tc = piece_of_rank[rank_of_tc]
    piece_of_pair = piece_of_tc[tc_of_pair]

    # CCs: (TC, column) with pairs; stats over the TC's pairs of that column
    cc_key = rank_of_tc[tc_of_pair] * SW + p_wl    # (TC rank, column)
    ucc, cc_of_pair = np.unique(cc_key, return_inverse=True)
    ncc = ucc.size
    cc_rank, cc_wl = ucc // SW, ucc % SW
    cc_piece = piece_of_rank[cc_rank]
    cc_dmin = np.full(ncc, 1 << 30)
    np.minimum.at(cc_dmin, cc_of_pair, p_d0)
    cc_hlo = np.full(ncc, 1 << 30)
    cc_hhi = np.full(ncc, -1)
    np.minimum.at(cc_hlo, cc_of_pair, p_h)
    np.maximum.at(cc_hhi, cc_of_pair, p_h)
    # CC order within piece: (column, dmin, TC in (strip, cell) order)
    cord = np.lexsort((tord[cc_rank], cc_dmin, cc_wl, cc_piece))
    pos_of_cc = np.empty(ncc, np.int64)
    pos_of_cc[cord] = np.arange(ncc)
    g_piece, g_wl = cc_piece[cord], cc_wl[cord]
    gstart = np.r_[True, (g_piece[1:] != g_piece[:-1]) | (g_wl[1:] != g_wl[:-1])]
    g_first = np.maximum.accumulate(np.where(gstart, np.arange(ncc), 0))
    q_in = np.arange(ncc) - g_first
    bhead = q_in % K == 0
    blk_of_pos = np.cumsum(bhead) - 1
    nblk = int(blk_of_pos[-1]) + 1 if ncc else 0
    b_pos0 = np.flatnonzero(bhead)
    b_piece, b_wl = g_piece[b_pos0], g_wl[b_pos0]
    # a block holds K CCs or the rest of its (piece, column) group
    gs = np.flatnonzero(gstart)
    g_end = np.repeat(np.r_[gs[1:], ncc], np.diff(np.r_[gs, ncc]))
    b_ncells = np.minimum(K, g_end[b_pos0] - b_pos0)
    k_of_pos = q_in % K
    hlo_sorted, hhi_sorted = cc_hlo[cord], cc_hhi[cord]
    b_hlo = np.minimum.reduceat(hlo_sorted, b_pos0) if nblk else np.zeros(0, np.int64)
    b_hhi = np.maximum.reduceat(hhi_sorted, b_pos0) if nblk else np.zeros(0, np.int64)
    b_nu = b_hhi - b_hlo + 1
    b_sz = K * b_nu
    # pieces: block ranges, entry bases within the piece
    pc_blk0 = np.searchsorted(b_piece, np.arange(npc), side="left")
    pc_nblk = np.diff(np.r_[pc_blk0, nblk])
    cum_b = np.cumsum(b_sz) - b_sz
    b_ebase = cum_b - cum_b[pc_blk0[b_piece]]
    pc_nent = np.add.reduceat(b_sz, pc_blk0) if npc else np.zeros(0, np.int64)
    pc_cc0 = np.searchsorted(g_piece, np.arange(npc), side="left")
    pc_ncc = np.diff(np.r_[pc_cc0, ncc])
    pc_tc0 = pc_rank0
    # CC table entry (in CC order): ebase + k | hlo << 16; block of each CC
    blk_of_cc = blk_of_pos[pos_of_cc]
    k_of_cc = k_of_pos[pos_of_cc]
    cc_tab = (b_ebase[blk_of_pos] + k_of_pos) | (b_hlo[blk_of_pos] << 16)
    # TC table (in TC rank order): destination and the partial rows of its
    # CCs, column by column (0xff: the TC has no pair in that column)
    tc_pr = np.full((ntc, SW), 0xFF, np.int64)
    blk_local = blk_of_cc - pc_blk0[cc_piece]
    tc_pr[cc_rank, cc_wl] = blk_local * K + k_of_cc
    # destinations: a cell with one TC is written directly, else one slot
    # per TC, numbered in (cell, strip) order
    corder = np.lexsort((tc_strip, tc_cell))
    c_sorted = tc_cell[corder]
    shared = np.zeros(ntc, dtype=bool)
    shared[1:] |= c_sorted[1:] == c_sorted[:-1]
    shared[:-1] |= c_sorted[1:] == c_sorted[:-1]
    slot_sorted = np.cumsum(shared) - shared
    nslots = int(shared.sum())
    dest_of_tc = np.empty(ntc, np.int64)
    dest_of_tc[corder] = np.where(shared, ~slot_sorted, c_sorted)
    tc_dest_rank = dest_of_tc[tord]
    comb_first = shared & np.r_[True, c_sorted[1:] != c_sorted[:-1]]
    comb_cell = c_sorted[comb_first]
    comb_slot0 = np.r_[slot_sorted[comb_first], nslots]
    occ = np.zeros(cells, dtype=bool)
    occ[tc_cell] = True
    empty = np.flatnonzero(~occ)
    n_occ_found = int(occ.sum())
    # pieces: pixel rows, depth range, records
    pc_plo = np.full(npc, 1 << 30)
    pc_phi = np.full(npc, -1)
    np.minimum.at(pc_plo, piece_of_pair, p_h)
    np.maximum.at(pc_phi, piece_of_pair, p_h)
    pc_dlo = np.full(npc, 1 << 30)
    pc_dhi = np.full(npc, -1)
    np.minimum.at(pc_dlo, piece_of_pair, p_d0)
    np.maximum.at(pc_dhi, piece_of_pair, p_d0 + p_n - 1)
    pc_nh = pc_phi - pc_plo + 1
    pc_nd = pc_dhi - pc_dlo + 1
    # records: pairs in (piece, local pixel, d0) order
    lp_piece = (p_h - pc_plo[piece_of_pair]) * SW + p_wl
    rord = np.lexsort((p_d0, lp_piece, piece_of_pair))
    r_piece = piece_of_pair[rord]
    pc_rec0 = np.searchsorted(r_piece, np.arange(npc), side="left")
    pc_nrec = np.diff(np.r_[pc_rec0, npairs])
    cc_local = pos_of_cc[cc_of_pair] - pc_cc0[piece_of_pair]
    rec = ((p_d0 - pc_dlo[piece_of_pair]) | ((p_n - 1) << 11) | (cc_local << 24))[rord]
    # per piece pixel table: first record of each local pixel (+ end)
    pc_npix = pc_nh * SW + 1
    pc_pix0 = np.cumsum(pc_npix) - pc_npix
    pixrec = np.zeros(int(pc_npix.sum()), np.int64)
    r_lp = lp_piece[rord]
    for j in range(npc):
        a, n = pc_rec0[j], pc_nrec[j]
        pixrec[pc_pix0[j]:pc_pix0[j] + pc_npix[j]] = np.searchsorted(
            r_lp[a:a + n], np.arange(pc_npix[j]), side="left")
    pc_ncol = np.minimum(SW, W - (pc_strip % nsw) * SW)
    assert np.all(rec >= 0) and np.all(pc_nd <= 2048) and np.all(p_n <= 8192)
    assert np.all(pc_nent <= ENT_BUDGET) and np.all(pc_ncc <= 256)

    # backward: the pairs in pixel-major order (stable by feature row)
    p_row = (bn[order][ph] * H + p_h) * W + (p_strip % nsw) * SW + p_wl
    bord = np.argsort(p_row, kind="stable")
    rows = B * N * H * W
    bp_cell = p_cell[bord]
    bp_dn = p_d0[bord] | (p_n[bord] << 16)
    pix_pair0 = np.searchsorted(p_row[bord], np.arange(rows + 1), side="left")

    piece = np.stack([pc_strip, pc_plo, pc_nh, pc_dlo, pc_nd, pc_blk0, pc_nblk, pc_rec0, pc_nrec,
                      pc_tc0, pc_ntc, pc_cc0, pc_ncc, pc_nent, pc_pix0, pc_ncol], axis=1) \
        if npc else np.zeros((0, PIECE_WORDS), np.int64)
    block = np.stack([b_wl | (b_ncells << 8), b_hlo, b_nu, b_ebase], axis=1) \
        if nblk else np.zeros((0, BLOCK_WORDS), np.int64)
    tc_tab = np.stack([tc_dest_rank, tc_pr[:, 0] | (tc_pr[:, 1] << 8) | (tc_pr[:, 2] << 16)
                       | (tc_pr[:, 3] << 24)], axis=1) if ntc else np.zeros((0, 2), np.int64)
    hdr = np.zeros(HDR_WORDS, np.int64)
    hdr[HDR["pairs"]] = npairs
    hdr[HDR["pieces"]] = npc
    hdr[HDR["blocks"]] = nblk
    hdr[HDR["valid"]] = nv
    hdr[HDR["occ"]] = int(plan["n_intervals"])
    hdr[HDR["occ_found"]] = n_occ_found
    hdr[HDR["empty"]] = empty.size
    hdr[HDR["slots"]] = nslots
    hdr[HDR["comb"]] = comb_cell.size
    hdr[HDR["tcs"]] = ntc
    hdr[HDR["ccs"]] = ncc
    hdr[HDR["max_ent"]] = int(pc_nent.max()) if npc else 0
    hdr[HDR["max_blk"]] = int(pc_nblk.max()) if npc else 0
    hdr[HDR["max_pix"]] = int((pc_npix - 1).max()) if npc else 0
    hdr[HDR["pixrec"]] = pixrec.size
    hdr[HDR["max_rec"]] = int(pc_nrec.max()) if npc else 0
    return dict(header=hdr, piece=piece, block=block, cc=cc_tab,
                tc=tc_tab, pixrec=pixrec, rec=rec, comb_cell=comb_cell, comb_slot0=comb_slot0,
                empty=empty, bp_cell=bp_cell, bp_dn=bp_dn, pix_pair0=pix_pair0,
                # for tests and the executor
                tcs_in_rank_order=dict(cell=tc_cell[tord], strip=tc_strip[tord]),
                pair_rd0=p_rd0, pair_n=p_n, shape=dict(shape))


def layout(shape: dict, n_valid: int, n_intervals: int) -> dict:
    """Word offsets and capacities of the device buffer (same rules as
    schedule_layout in the library)."""
    B, N, H, W = (int(shape[k]) for k in "BNHW")
    cells = B * int(shape["Z"]) * int(shape["Y"]) * int(shape["X"])
    rows = B * N * H * W
    nv = max(n_valid, 1)
    n_empty = max(cells - n_intervals, 0)
    strips = B * N * (-(-W // SW))
    pcap = min(nv, 2 * strips + nv // max(tc_max(H), 1) + nv // PAIRS + 2)
    sizes = [("header", HDR_WORDS), ("piece", PIECE_WORDS * pcap), ("block", BLOCK_WORDS * nv),
             ("cc", nv), ("tc", 2 * nv), ("pixrec", pcap * (H * SW + 1)), ("rec", nv),
             ("comb_cell", n_intervals + 1), ("comb_slot0", n_intervals + 1),
             ("empty", n_empty + 1), ("bp_cell", nv), ("bp_dn", nv), ("pix_pair0", rows + 1)]
    off, out = 0, {}
    for name, n in sizes:
        out[name] = (off // 4, n)
        off += -(-4 * n // ALIGN) * ALIGN
    out["total"] = off
    return out


def pack(s: dict, n_valid: int, n_intervals: int) -> np.ndarray:
    """The device buffer (bytes) of a derived schedule."""
    lay = layout(s["shape"], n_valid, n_intervals)
    buf = np.zeros(lay["total"] // 4, np.uint32)
    assert buf.size * 4 == lay["total"]
    total = lay.pop("total")
    for name, (off, cap) in lay.items():
        a = np.asarray(s[name]).reshape(-1).astype(np.int64)
        assert a.size <= cap, (name, a.size, cap)
        buf[off:off + a.size] = (a & 0xFFFFFFFF).astype(np.uint32)
    return buf.view(np.uint8)


def decode(buf: np.ndarray, shape: dict, n_valid: int, n_intervals: int) -> dict:
    """Arrays of a device buffer, trimmed to the header's counts."""
    w = buf.view(np.int32)
    lay = layout(shape, n_valid, n_intervals)
    hdr = w[:HDR_WORDS].astype(np.int64)
    n = {k: int(hdr[i]) for k, i in HDR.items()}

    def arr(name, count, width=1):
        off, _ = lay[name]
        a = w[off:off + count * width].astype(np.int64)
        return a.reshape(count, width) if width > 1 else a

    rows = int(shape["B"]) * int(shape["N"]) * int(shape["H"]) * int(shape["W"])
    u = lambda a: a & 0xFFFFFFFF
    return dict(header=hdr, piece=arr("piece", n["pieces"], PIECE_WORDS),
                block=arr("block", n["blocks"], BLOCK_WORDS), cc=arr("cc", n["ccs"]),
                tc=np.stack([arr("tc", n["tcs"], 2)[:, 0], u(arr("tc", n["tcs"], 2)[:, 1])], axis=1)
                if n["tcs"] else np.zeros((0, 2), np.int64),
                pixrec=arr("pixrec", n["pixrec"]), rec=u(arr("rec", n["pairs"])),
                comb_cell=arr("comb_cell", n["comb"]), comb_slot0=arr("comb_slot0", n["comb"] + 1),
                empty=arr("empty", n["empty"]), bp_cell=arr("bp_cell", n["pairs"]),
                bp_dn=u(arr("bp_dn", n["pairs"])), pix_pair0=arr("pix_pair0", rows + 1))


def execute(s: dict, depth: np.ndarray, feat: np.ndarray) -> np.ndarray:
    """The scheduled forward in float64, in the order the kernels use the
    schedule: per piece, dense weights from the depth runs of its records,
    per block the weights times the column's feature rows, per TC the sum of
    its column partials, then the cross-strip sum of slots."""
    sh = s["shape"]
    B, N, D, H, W, C, X, Y, Z = (int(sh[k]) for k in "BNDHWCXYZ")
    nsw = -(-W // SW)
    HW = H * W
    dep = depth.reshape(-1).astype(np.float64)
    fea = feat.reshape(-1, C).astype(np.float64)
    out = np.zeros((B * Z * Y * X, C))
    slots = np.zeros((int(s["header"][HDR["slots"]]), C))
    for pc in s["piece"]:
        strip, plo, nh, dlo, nd, blk0, nblk, rec0, nrec, tc0, ntc, cc0, ncc, nent, pix0, ncol = pc
        bn, w0 = strip // nsw, (strip % nsw) * SW
        wts = np.zeros(nent)
        for lp in range(nh * SW):
            hh, wl = plo + lp // SW, lp % SW
            for r in s["rec"][rec0 + s["pixrec"][pix0 + lp]:rec0 + s["pixrec"][pix0 + lp + 1]]:
                d0 = dlo + (r & 0x7FF)
                n = ((r >> 11) & 0x1FFF) + 1
                cc = s["cc"][cc0 + (r >> 24)]
                e = (cc & 0xFFFF) + (hh - (cc >> 16)) * K
                p = ((bn * D + d0 + np.arange(n)) * H + hh) * W + w0 + wl
                wts[e] += dep[p].sum()
        part = np.zeros((nblk * K, C))
        for j in range(nblk):
            wlc_cells, hlo, nu, eb = s["block"][blk0 + j]
            wl = wlc_cells & 0xFF
            rows_ = (bn * H + hlo + np.arange(nu)) * W + w0 + wl
            wmat = wts[eb:eb + nu * K].reshape(nu, K)
            part[j * K:(j + 1) * K] = wmat.T @ fea[rows_]
        for t in range(ntc):
            dest, prs = s["tc"][tc0 + t]
            acc = np.zeros(C)
            for c in range(SW):
                pr = (prs >> (8 * c)) & 0xFF
                if pr != 0xFF:
                    acc += part[pr]
            if dest >= 0:
                out[dest] = acc
            else:
                slots[~dest] = acc
    for m, cell in enumerate(s["comb_cell"]):
        out[cell] = slots[s["comb_slot0"][m]:s["comb_slot0"][m + 1]].sum(axis=0)
    return out.reshape(B, Z, Y, X, C)

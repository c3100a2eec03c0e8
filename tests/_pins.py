"""Independent checks that pin the CPU oracle to the paper and to mathematics.

Nothing here calls the oracle's own helpers: brute force walks the frustum
points with nested loops and indexes the BEV output as a (B, Z, Y, X, C)
array, library routines (``np.ravel_multi_index``, ``np.bincount``, Python's
``sorted``) stand in for the rank arithmetic, and closed forms (mass
conservation, one-hot reductions, adjoint identity, exact finite
differences of a bilinear map) check the results.  Each ``check_*`` returns a
list of failure messages so that tests can also confirm that a deliberately
broken oracle is caught.
"""

from __future__ import annotations

import numpy as np


def dims(shape):
    return tuple(int(shape[k]) for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z"))


# ----------------------------------------------------------------------------
# brute force, pure Python loops (tiny inputs only)
# ----------------------------------------------------------------------------

def _walk(shape, coor):
    """Yield (b, n, d, h, w, p, inside, (x, y, z)) for every frustum point in
    depth-score order, counting p as it goes."""
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    p = 0
    for b in range(B):
        for n in range(N):
            for d in range(D):
                for h in range(H):
                    for w in range(W):
                        x, y, z = (int(v) for v in coor[p])
                        inside = 0 <= x < X and 0 <= y < Y and 0 <= z < Z
                        yield b, n, d, h, w, p, inside, (x, y, z)
                        p += 1


def brute_prepare(coor, shape):
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    kept = []
    for b, n, d, h, w, p, inside, (x, y, z) in _walk(shape, coor):
        if inside:
            cell = int(np.ravel_multi_index((b, z, y, x), (B, Z, Y, X)))
            row = int(np.ravel_multi_index((b, n, h, w), (B, N, H, W)))
            kept.append(((b, z, y, x), p, row, cell))
    kept = sorted(kept, key=lambda t: (t[0], t[1]))
    rd = [t[1] for t in kept]
    rf = [t[2] for t in kept]
    rb = [t[3] for t in kept]
    starts, lengths = [], []
    for i, cell in enumerate(rb):
        if i == 0 or cell != rb[i - 1]:
            starts.append(i)
            lengths.append(1)
        else:
            lengths[-1] += 1
    return {"ranks_depth": rd, "ranks_feat": rf, "ranks_bev": rb,
            "interval_starts": starts, "interval_lengths": lengths,
            "n_valid": len(rd), "n_intervals": len(starts)}


def brute_forward(depth, feat, coor, shape):
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    out = np.zeros((B, Z, Y, X, C))
    for b, n, d, h, w, p, inside, (x, y, z) in _walk(shape, coor):
        if inside:
            for c in range(C):
                out[b, z, y, x, c] += float(depth[b, n, d, h, w]) * float(feat[b, n, h, w, c])
    return out


def brute_backward(grad_out, depth, feat, coor, shape):
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    gd = np.zeros((B, N, D, H, W))
    gf = np.zeros((B, N, H, W, C))
    for b, n, d, h, w, p, inside, (x, y, z) in _walk(shape, coor):
        if inside:
            s = 0.0
            for c in range(C):
                s += float(grad_out[b, z, y, x, c]) * float(feat[b, n, h, w, c])
                gf[b, n, h, w, c] += float(depth[b, n, d, h, w]) * float(grad_out[b, z, y, x, c])
            gd[b, n, d, h, w] = s
    return gd, gf


# ----------------------------------------------------------------------------
# checks
# ----------------------------------------------------------------------------

def _close(a, b, scale, rel=1e-12):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return bool(np.all(np.abs(a - b) <= rel * (np.abs(scale) + 1.0)))


def check_prepare_brute(prepare_fn, coor, shape):
    fails = []
    ref = brute_prepare(coor, shape)
    got = prepare_fn(coor, shape)
    for key in ("ranks_depth", "ranks_feat", "ranks_bev", "interval_starts", "interval_lengths"):
        if not np.array_equal(np.asarray(got[key], dtype=np.int64), np.asarray(ref[key], dtype=np.int64)):
            fails.append(f"prepare {key} differs from brute force")
    for key in ("n_valid", "n_intervals"):
        if int(got[key]) != int(ref[key]):
            fails.append(f"prepare {key} {got[key]} != {ref[key]}")
    return fails


def check_prepare_invariants(prepare_fn, coor, shape):
    """Counting-sort identity and sortedness invariants (any size)."""
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    fails = []
    got = prepare_fn(coor, shape)
    rd = np.asarray(got["ranks_depth"], dtype=np.int64)
    rf = np.asarray(got["ranks_feat"], dtype=np.int64)
    rb = np.asarray(got["ranks_bev"], dtype=np.int64)
    st = np.asarray(got["interval_starts"], dtype=np.int64)
    ln = np.asarray(got["interval_lengths"], dtype=np.int64)
    x, y, z = (coor[:, i].astype(np.int64) for i in range(3))
    inside = (x >= 0) & (x < X) & (y >= 0) & (y < Y) & (z >= 0) & (z < Z)
    pts = np.flatnonzero(inside)
    b_of = pts // (N * D * H * W)
    cells_all = np.ravel_multi_index((b_of, z[pts], y[pts], x[pts]), (B, Z, Y, X))
    if rd.size != pts.size or int(got["n_valid"]) != pts.size:
        fails.append("n_valid differs from the in-grid count")
        return fails
    # set equality of (rank_depth, rank_bev) with the in-grid points
    if not np.array_equal(np.sort(rd), pts):
        fails.append("ranks_depth is not a permutation of the in-grid points")
    if not np.array_equal(rb[np.argsort(rd)], cells_all):
        fails.append("ranks_bev does not match each point's voxel")
    unr = np.unravel_index(rd, (B, N, D, H, W))
    if not np.array_equal(rf, np.ravel_multi_index((unr[0], unr[1], unr[3], unr[4]), (B, N, H, W))):
        fails.append("ranks_feat does not name each point's image-feature row")
    if rb.size and np.any(np.diff(rb) < 0):
        fails.append("ranks_bev not sorted")
    same = np.diff(rb) == 0
    if rd.size and np.any(np.diff(rd)[same] <= 0):
        fails.append("ties not in ascending frustum index (sort not stable)")
    counts = np.bincount(cells_all, minlength=B * Z * Y * X)
    occ = np.flatnonzero(counts)
    if not np.array_equal(ln, counts[occ]):
        fails.append("interval lengths differ from the voxel histogram")
    if not np.array_equal(st, np.concatenate([[0], np.cumsum(counts[occ])[:-1]]) if occ.size else st):
        fails.append("interval starts differ from the histogram's exclusive sum")
    if int(ln.sum()) != pts.size:
        fails.append("interval lengths do not sum to n_valid")
    if int(got["n_intervals"]) != occ.size:
        fails.append("n_intervals differs from the number of occupied voxels")
    return fails


def check_forward_brute(forward_fn, depth, feat, coor, shape):
    out, mag = forward_fn(depth, feat, coor, shape)
    ref = brute_forward(depth, feat, coor, shape)
    fails = []
    if out.shape != ref.shape:
        return [f"forward shape {out.shape} != {ref.shape}"]
    if not _close(out, ref, mag):
        fails.append("forward differs from brute force")
    ref_mag = brute_forward(np.abs(depth.astype(np.float64)), np.abs(feat.astype(np.float64)), coor, shape)
    if not _close(mag, ref_mag, ref_mag):
        fails.append("forward |terms| differs from brute force")
    return fails


def check_forward_identities(forward_fn, depth, feat, coor, shape):
    """Mass conservation, all-ones counts, one-hot depth scatter, linearity."""
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    fails = []
    x, y, z = (coor[:, i].astype(np.int64) for i in range(3))
    inside = (x >= 0) & (x < X) & (y >= 0) & (y < Y) & (z >= 0) & (z < Z)
    inside5 = inside.reshape(B, N, D, H, W)
    dep = depth.astype(np.float64)
    img = feat.astype(np.float64)
    out, mag = forward_fn(depth, feat, coor, shape)

    # (1) mass conservation per channel
    mass = np.einsum("bndhw,bnhwc->c", dep * inside5, img)
    if not _close(out.reshape(-1, C).sum(axis=0), mass, mag.reshape(-1, C).sum(axis=0), rel=1e-10):
        fails.append("mass not conserved")

    # (2) all-ones: every cell holds its point count, in every channel
    pts = np.flatnonzero(inside)
    cells_all = np.ravel_multi_index((pts // (N * D * H * W), z[pts], y[pts], x[pts]), (B, Z, Y, X))
    counts = np.bincount(cells_all, minlength=B * Z * Y * X).astype(np.float64)
    ones_out, _ = forward_fn(np.ones_like(dep), np.ones_like(img), coor, shape)
    if not np.array_equal(ones_out.reshape(-1, C), np.repeat(counts[:, None], C, axis=1)):
        fails.append("all-ones forward differs from the voxel point counts")

    # (3) one-hot depth: the forward is a plain scatter of feature rows
    rng = np.random.default_rng(123)
    k = rng.integers(0, D, size=(B, N, H, W))
    onehot = (np.arange(D)[None, None, :, None, None] == k[:, :, None, :, :]).astype(np.float64)
    oh_out, _ = forward_fn(onehot, img, coor, shape)
    bb, nn, hh, ww = np.meshgrid(np.arange(B), np.arange(N), np.arange(H), np.arange(W), indexing="ij")
    pp = np.ravel_multi_index((bb, nn, k, hh, ww), (B, N, D, H, W)).ravel()
    rows = np.ravel_multi_index((bb, nn, hh, ww), (B, N, H, W)).ravel()
    sel = inside[pp]
    cell_of = np.ravel_multi_index((bb.ravel()[sel], z[pp[sel]], y[pp[sel]], x[pp[sel]]), (B, Z, Y, X))
    scatter = np.stack([np.bincount(cell_of, weights=img.reshape(-1, C)[rows[sel], c],
                                    minlength=B * Z * Y * X) for c in range(C)], axis=1)
    if not _close(oh_out.reshape(-1, C), scatter, np.abs(scatter) + 1.0, rel=1e-12):
        fails.append("one-hot depth forward differs from a plain feature scatter")

    # (4) linearity in the depth score
    d2 = rng.standard_normal(dep.shape)
    a = 0.37
    lin_out, lin_mag = forward_fn(a * dep + d2, img, coor, shape)
    o2, m2 = forward_fn(d2, img, coor, shape)
    if not _close(lin_out, a * out + o2, lin_mag + m2 + mag, rel=1e-12):
        fails.append("forward not linear in the depth score")
    return fails


def check_backward_brute(backward_fn, grad_out, depth, feat, coor, shape):
    gd, gf, gd_mag, gf_mag = backward_fn(grad_out, depth, feat, coor, shape)
    rgd, rgf = brute_backward(grad_out, depth, feat, coor, shape)
    fails = []
    if not _close(gd, rgd, gd_mag):
        fails.append("grad_depth differs from brute force")
    if not _close(gf, rgf, gf_mag):
        fails.append("grad_feat differs from brute force")
    return fails


def check_backward_identities(backward_fn, forward_fn, grad_out, depth, feat, coor, shape,
                              n_fd: int = 12):
    """Adjoint identity, exact central differences, one-hot reductions."""
    B, N, D, H, W, C, X, Y, Z = dims(shape)
    fails = []
    g = grad_out.astype(np.float64)
    dep = depth.astype(np.float64)
    img = feat.astype(np.float64)
    gd, gf, gd_mag, gf_mag = backward_fn(grad_out, depth, feat, coor, shape)
    out, mag = forward_fn(depth, feat, coor, shape)

    # (1) adjoint identity: <g, out> = <gd, depth> = <gf, feat>
    tri = float(np.sum(g * out))
    scale = float(np.sum(np.abs(g) * mag)) + 1.0
    if abs(tri - float(np.sum(gd * dep))) > 1e-10 * scale:
        fails.append("adjoint identity <g,out> = <grad_depth,depth> violated")
    if abs(tri - float(np.sum(gf * img))) > 1e-10 * scale:
        fails.append("adjoint identity <g,out> = <grad_feat,feat> violated")

    # (2) central differences: L = <g, out> is linear in depth and in feat,
    # so the difference quotient is exact up to rounding for any step.
    rng = np.random.default_rng(7)
    def loss(dv, fv):
        o, _ = forward_fn(dv, fv, coor, shape)
        return float(np.sum(g * o))
    for _ in range(n_fd):
        i = tuple(int(rng.integers(0, s)) for s in dep.shape)
        step = 0.5
        dp = dep.copy(); dp[i] += step
        dm = dep.copy(); dm[i] -= step
        fd = (loss(dp, img) - loss(dm, img)) / (2 * step)
        if abs(fd - gd[i]) > 1e-9 * (scale + abs(fd)):
            fails.append(f"grad_depth{i} != central difference")
            break
    for _ in range(n_fd):
        i = tuple(int(rng.integers(0, s)) for s in img.shape)
        step = 0.5
        fp = img.copy(); fp[i] += step
        fm = img.copy(); fm[i] -= step
        fd = (loss(dep, fp) - loss(dep, fm)) / (2 * step)
        if abs(fd - gf[i]) > 1e-9 * (scale + abs(fd)):
            fails.append(f"grad_feat{i} != central difference")
            break

    # (3) one-hot channel feature: grad_depth picks that channel of grad_out
    x, y, z = (coor[:, j].astype(np.int64) for j in range(3))
    inside = (x >= 0) & (x < X) & (y >= 0) & (y < Y) & (z >= 0) & (z < Z)
    c0 = C // 2
    e = np.zeros_like(img); e[..., c0] = 1.0
    gd_e, _, _, _ = backward_fn(grad_out, depth, e, coor, shape)
    p = np.arange(B * N * D * H * W)
    want = np.zeros(p.size)
    pi = p[inside]
    want[inside] = g[pi // (N * D * H * W), z[inside], y[inside], x[inside], c0]
    if not np.array_equal(gd_e.reshape(-1), want):
        fails.append("one-hot channel feature: grad_depth != grad_out channel")

    # (4) one-hot depth: grad_feat of a pixel is grad_out of its chosen voxel
    k = rng.integers(0, D, size=(B, N, H, W))
    onehot = (np.arange(D)[None, None, :, None, None] == k[:, :, None, :, :]).astype(np.float64)
    _, gf_o, _, _ = backward_fn(grad_out, onehot, feat, coor, shape)
    bb, nn, hh, ww = np.meshgrid(np.arange(B), np.arange(N), np.arange(H), np.arange(W), indexing="ij")
    pp = np.ravel_multi_index((bb, nn, k, hh, ww), (B, N, D, H, W))
    want_f = np.zeros((B, N, H, W, C))
    ok = inside[pp]
    want_f[ok] = g[bb[ok], z[pp[ok]], y[pp[ok]], x[pp[ok]]]
    if not np.array_equal(gf_o, want_f):
        fails.append("one-hot depth: grad_feat != grad_out row of the chosen voxel")

    # (5) dropped points get exactly zero depth gradient
    if np.any(gd.reshape(-1)[~inside] != 0.0):
        fails.append("dropped points have non-zero grad_depth")
    return fails

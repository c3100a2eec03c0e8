"""Float64 reference of the BEVPoolv2 view transformation (test infrastructure).

Everything here follows the Lift-Splat-Shoot definition restated in
BEVPoolv2 section 2.1, paragraph 1:

* the frustum feature of shape (N, D, H, W, C) is the depth score
  (N, D, H, W) times the image feature (N, H, W, C), broadcast over D and C;
* each frustum point carries a voxel index computed offline from the camera
  intrinsics and extrinsics (here: the int32 (P, 3) array ``coor``);
* frustum points outside the scope of every voxel are filtered out;
* the remaining points are sorted by voxel index and the points that share a
  voxel are summed.

Section 2.1, paragraph 2 (BEVPoolv2 proper) keeps the same result but carries
each point's frustum index through the preprocessing instead of the
materialised feature; ``prepare_ref`` is that preprocessing.  The backward
pass is not described by the paper; ``backward_ref`` is the chain rule
through the materialised frustum feature.

Conventions (the paper leaves them open):
* points are enumerated p = (((b*N + n)*D + d)*H + h)*W + w, the depth-score
  layout with a leading batch axis; the depth rank of a point is p itself;
* the feature rank is the image-feature row ((b*N + n)*H + h)*W + w;
* the BEV rank is ((b*Z + z)*Y + y)*X + x and the output is (B, Z, Y, X, C);
* "sorting by voxel index" is read as a stable sort, so ties keep ascending
  frustum index;
* every output element also gets the sum of the absolute values of the terms
  that make it up, which scales the floating-point tolerance.

Inputs of reduced precision are converted exactly to float64 first.
"""

from __future__ import annotations

import numpy as np

_F64 = np.float64


def _dims(shape: dict):
    return tuple(int(shape[k]) for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z"))


def kept_mask(coor: np.ndarray, shape: dict) -> np.ndarray:
    """Section 2.1: a frustum point is kept when its voxel index lies inside
    the grid, 0 <= x < X, 0 <= y < Y, 0 <= z < Z."""
    _, _, _, _, _, _, X, Y, Z = _dims(shape)
    x = coor[:, 0].astype(np.int64)
    y = coor[:, 1].astype(np.int64)
    z = coor[:, 2].astype(np.int64)
    return (x >= 0) & (x < X) & (y >= 0) & (y < Y) & (z >= 0) & (z < Z)


def point_ranks(p: np.ndarray, coor_p: np.ndarray, shape: dict):
    """Depth rank, feature rank and BEV rank of frustum points ``p``.

    ``coor_p`` holds the (x, y, z) voxel index of each of those points.
    """
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    p = p.astype(np.int64)
    w = p % W
    h = (p // W) % H
    bn = p // (W * H * D)          # b*N + n
    rank_depth = p
    rank_feat = (bn * H + h) * W + w
    b = bn // N
    x = coor_p[:, 0].astype(np.int64)
    y = coor_p[:, 1].astype(np.int64)
    z = coor_p[:, 2].astype(np.int64)
    rank_bev = ((b * Z + z) * Y + y) * X + x
    return rank_depth, rank_feat, rank_bev


def prepare_ref(coor: np.ndarray, shape: dict) -> dict:
    """Preprocessing of section 2.1: filter, sort by voxel index, intervals.

    Returns int32 arrays ranks_depth, ranks_feat, ranks_bev (length n_valid,
    sorted by BEV rank, ties in ascending frustum index), interval_starts and
    interval_lengths (one entry per occupied BEV cell, in ascending cell
    order), and the counts n_valid and n_intervals.
    """
    kept = kept_mask(coor, shape)
    p = np.flatnonzero(kept)
    rd, rf, rb = point_ranks(p, coor[p], shape)
    order = np.argsort(rb, kind="stable")
    rd, rf, rb = rd[order], rf[order], rb[order]
    _, starts, lengths = np.unique(rb, return_index=True, return_counts=True)
    return {
        "ranks_depth": rd.astype(np.int32),
        "ranks_feat": rf.astype(np.int32),
        "ranks_bev": rb.astype(np.int32),
        "interval_starts": starts.astype(np.int32),
        "interval_lengths": lengths.astype(np.int32),
        "n_valid": int(p.size),
        "n_intervals": int(starts.size),
    }


def frustum_feature(depth: np.ndarray, feat: np.ndarray, b: int, n: int) -> np.ndarray:
    """(D, H, W, C) frustum feature of view n in sample b: the depth score
    times the image feature (section 2.1, paragraph 1)."""
    dep = depth[b, n].astype(_F64)        # (D, H, W)
    img = feat[b, n].astype(_F64)         # (H, W, C)
    return dep[:, :, :, None] * img[None, :, :, :]


def _view_points(b: int, n: int, shape: dict) -> np.ndarray:
    B, N, D, H, W, *_ = _dims(shape)
    per_view = D * H * W
    base = (b * N + n) * per_view
    return np.arange(base, base + per_view, dtype=np.int64)


def forward_ref(depth: np.ndarray, feat: np.ndarray, coor: np.ndarray, shape: dict):
    """BEV feature (B, Z, Y, X, C) and the matching sum of |terms|.

    Materialises the frustum feature one view at a time, drops points outside
    the grid and scatter-adds the rest into their voxel.  Cells no point
    reaches are exactly zero.
    """
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    cells = B * Z * Y * X
    out = np.zeros((cells, C), dtype=_F64)
    mag = np.zeros((cells, C), dtype=_F64)
    for b in range(B):
        for n in range(N):
            frustum = frustum_feature(depth, feat, b, n).reshape(D * H * W, C)
            p = _view_points(b, n, shape)
            c = coor[p]
            kept = kept_mask(c, shape)
            _, _, rb = point_ranks(p[kept], c[kept], shape)
            np.add.at(out, rb, frustum[kept])
            np.add.at(mag, rb, np.abs(frustum[kept]))
    return out.reshape(B, Z, Y, X, C), mag.reshape(B, Z, Y, X, C)


def backward_ref(grad_out: np.ndarray, depth: np.ndarray, feat: np.ndarray,
                 coor: np.ndarray, shape: dict):
    """Gradients of the forward with respect to the depth score and feature.

    Chain rule through the frustum feature F = depth x feat: the gradient
    reaching F[p, :] is the upstream gradient row of p's voxel when p is kept
    and zero otherwise; then dL/ddepth[d,h,w] = sum_c dL/dF[d,h,w,c]*feat[h,w,c]
    and dL/dfeat[h,w,c] = sum_d dL/dF[d,h,w,c]*depth[d,h,w].

    Returns grad_depth (B,N,D,H,W), grad_feat (B,N,H,W,C) and their |terms|
    sums, all float64.
    """
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    g = grad_out.reshape(B * Z * Y * X, C).astype(_F64)
    gd = np.zeros((B, N, D, H, W), dtype=_F64)
    gd_mag = np.zeros_like(gd)
    gf = np.zeros((B, N, H, W, C), dtype=_F64)
    gf_mag = np.zeros_like(gf)
    for b in range(B):
        for n in range(N):
            dep = depth[b, n].astype(_F64)
            img = feat[b, n].astype(_F64)
            p = _view_points(b, n, shape)
            c = coor[p]
            kept = kept_mask(c, shape)
            _, _, rb = point_ranks(p[kept], c[kept], shape)
            dF = np.zeros((D * H * W, C), dtype=_F64)
            dF[kept] = g[rb]
            dF = dF.reshape(D, H, W, C)
            t_depth = dF * img[None, :, :, :]
            gd[b, n] = t_depth.sum(axis=3)
            gd_mag[b, n] = np.abs(t_depth).sum(axis=3)
            t_feat = dF * dep[:, :, :, None]
            gf[b, n] = t_feat.sum(axis=0)
            gf_mag[b, n] = np.abs(t_feat).sum(axis=0)
    return gd, gf, gd_mag, gf_mag


# ---------------------------------------------------------------------------
# Sampled forms: the same definitions evaluated for a chosen subset of output
# elements, for workloads too large to run the full reference in a test.
# ---------------------------------------------------------------------------

def forward_cells_ref(depth: np.ndarray, feat: np.ndarray, coor: np.ndarray,
                      shape: dict, cells: np.ndarray):
    """Rows ``cells`` of the flattened (B*Z*Y*X, C) BEV output, and |terms|."""
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    cells = np.asarray(cells, dtype=np.int64)
    kept = kept_mask(coor, shape)
    p = np.flatnonzero(kept)
    rd, rf, rb = point_ranks(p, coor[p], shape)
    sel = np.isin(rb, cells)
    rd, rf, rb = rd[sel], rf[sel], rb[sel]
    terms = (depth.reshape(-1)[rd].astype(_F64)[:, None]
             * feat.reshape(-1, C)[rf].astype(_F64))
    row_of = {int(cell): i for i, cell in enumerate(cells)}
    rows = np.fromiter((row_of[int(r)] for r in rb), dtype=np.int64, count=rb.size)
    out = np.zeros((cells.size, C), dtype=_F64)
    mag = np.zeros((cells.size, C), dtype=_F64)
    np.add.at(out, rows, terms)
    np.add.at(mag, rows, np.abs(terms))
    return out, mag


def grad_depth_points_ref(grad_out: np.ndarray, feat: np.ndarray, coor: np.ndarray,
                          shape: dict, points: np.ndarray):
    """grad_depth at frustum indices ``points`` (flattened), and |terms|."""
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    points = np.asarray(points, dtype=np.int64)
    g = grad_out.reshape(-1, C)
    img = feat.reshape(-1, C)
    c = coor[points]
    kept = kept_mask(c, shape)
    _, rf, rb = point_ranks(points, c, shape)
    val = np.zeros(points.size, dtype=_F64)
    mag = np.zeros(points.size, dtype=_F64)
    for i in np.flatnonzero(kept):
        t = g[rb[i]].astype(_F64) * img[rf[i]].astype(_F64)
        val[i] = t.sum()
        mag[i] = np.abs(t).sum()
    return val, mag


def grad_feat_pixels_ref(grad_out: np.ndarray, depth: np.ndarray, coor: np.ndarray,
                         shape: dict, pixels: np.ndarray):
    """grad_feat rows at feature ranks ``pixels`` ((b*N+n)*H+h)*W+w, and |terms|."""
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    pixels = np.asarray(pixels, dtype=np.int64)
    g = grad_out.reshape(-1, C)
    dep = depth.reshape(-1)
    val = np.zeros((pixels.size, C), dtype=_F64)
    mag = np.zeros((pixels.size, C), dtype=_F64)
    for i, f in enumerate(pixels):
        bn, hw = divmod(int(f), H * W)
        pts = (bn * D + np.arange(D, dtype=np.int64)) * (H * W) + hw
        c = coor[pts]
        kept = kept_mask(c, shape)
        _, _, rb = point_ranks(pts[kept], c[kept], shape)
        t = dep[pts[kept]].astype(_F64)[:, None] * g[rb].astype(_F64)
        val[i] = t.sum(axis=0)
        mag[i] = np.abs(t).sum(axis=0)
    return val, mag


# ---- depth scores from logits (the fused depth-softmax forward) -----------
#
# Section 2.1, paragraph 1 takes the depth score (N, D, H, W) as each pixel's
# distribution over its D depth classes.  When a network gives logits, the
# distribution is their softmax over the depth axis.  The reading here: the
# softmax is taken per (b, n, h, w) over d, in float64 from the given
# (possibly rounded) logits, and the forward is then exactly forward_ref on
# those scores.


def depth_lse_ref(logits: np.ndarray) -> np.ndarray:
    """Log-sum-exp over the depth axis of logits (B, N, D, H, W): (B, N, H, W).

    Computed as m + log(sum exp(logit - m)) with m the largest logit of the
    pixel, so no term overflows."""
    x = np.asarray(logits, dtype=_F64)
    m = x.max(axis=2, keepdims=True)
    return (m + np.log(np.exp(x - m).sum(axis=2, keepdims=True)))[:, :, 0]


def depth_softmax_ref(logits: np.ndarray) -> np.ndarray:
    """Depth scores exp(logit - lse) (B, N, D, H, W): per pixel, a
    distribution over the depth bins."""
    x = np.asarray(logits, dtype=_F64)
    return np.exp(x - depth_lse_ref(x)[:, :, None])


def forward_softmax_ref(logits: np.ndarray, feat: np.ndarray, coor: np.ndarray, shape: dict):
    """forward_ref with the depth scores of depth_softmax_ref(logits)."""
    return forward_ref(depth_softmax_ref(logits), feat, coor, shape)


# ---- voxel index from camera parameters (the on-device geometry) ----------
#
# Section 2.1 takes each frustum point's voxel index as computed offline from
# the camera intrinsics and extrinsics.  The reading here (a pinhole model):
# feature cell (h, w) looks through the pixel centre (u, v) = ((w + 0.5) s,
# (h + 0.5) s) for stride s; depth bin k lies at depth_start + k depth_step
# along the optical axis; the camera point is ((u - cx) dep / fx,
# (v - cy) dep / fy, dep); the ego point is R @ cam + t, each coordinate
# summed in the order (R0 X + R1 Y) + R2 Z + t; the voxel index is
# floor((e - lo) / res), clipped to +-2^30 so it stays representable; points
# outside the grid keep their index (the filter of prepare drops them).


def geometry_ref(cams: np.ndarray, params: dict, shape: dict) -> np.ndarray:
    """int32 (B*N*D*H*W, 3) voxel index (x, y, z) of every frustum point
    from per-camera parameters cams (B, N, 16): fx, fy, cx, cy, R (3x3,
    row-major), t."""
    B, N, D, H, W, C, X, Y, Z = _dims(shape)
    cams = np.asarray(cams, dtype=_F64)
    s = _F64(params["stride"])
    u = (np.arange(W, dtype=_F64) + 0.5) * s
    v = (np.arange(H, dtype=_F64) + 0.5) * s
    dep = _F64(params["depth_start"]) + np.arange(D, dtype=_F64) * _F64(params["depth_step"])
    lo = np.asarray(params["lo"], dtype=_F64)
    res = np.asarray(params["res"], dtype=_F64)
    out = np.empty((B, N, D, H, W, 3), dtype=np.int64)
    d3 = dep[:, None, None]
    for b in range(B):
        for n in range(N):
            fx, fy, cx, cy = cams[b, n, :4]
            R = cams[b, n, 4:13].reshape(3, 3)
            t = cams[b, n, 13:16]
            Xc = np.broadcast_to(((u[None, None, :] - cx) * d3) / fx, (D, H, W))
            Yc = np.broadcast_to(((v[None, :, None] - cy) * d3) / fy, (D, H, W))
            Zc = np.broadcast_to(d3, (D, H, W))
            for i in range(3):
                e = ((R[i, 0] * Xc + R[i, 1] * Yc) + R[i, 2] * Zc) + t[i]
                idx = np.floor((e - lo[i]) / res[i])
                out[b, n, ..., i] = np.clip(idx, -(2 ** 30), 2 ** 30).astype(np.int64)
    return out.reshape(-1, 3).astype(np.int32)

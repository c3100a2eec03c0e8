"""Seeded activations: depth score, image feature and upstream gradient.

Distributions (the paper's trained networks are not available):
* image feature ~ N(0, 1);
* depth score = softmax over the D depth classes of 3*N(0, 1) logits,
  computed in float64 and then rounded to the working precision -- the depth
  score in section 2.1 is a per-pixel distribution over depth classes;
* upstream gradient of the BEV output ~ N(0, 1).

Draw order with ``numpy.random.default_rng(seed)``: for each sample b in
turn, the logits (N, D, H, W), then the feature (N, H, W, C), then the
gradient (Z, Y, X, C).  Casts to float32/float16 round to nearest even.
"""

from __future__ import annotations

import numpy as np

from .configs import Config

_NP_DTYPE = {"f32": np.float32, "f16": np.float16}


def np_dtype(name: str):
    return _NP_DTYPE[name]


def _softmax_depth(logits: np.ndarray) -> np.ndarray:
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=1, keepdims=True)


def draw_inputs(cfg: Config, seed: int | None = None, with_grad: bool = True,
                with_logits: bool = False) -> dict:
    """Depth (B,N,D,H,W), feat (B,N,H,W,C) and grad_out (B,Z,Y,X,C); with
    with_logits also the depth logits (B,N,D,H,W) the scores were drawn
    from, rounded to the working precision."""
    rng = np.random.default_rng(cfg.seed if seed is None else seed)
    dt = _NP_DTYPE[cfg.dtype]
    odt = _NP_DTYPE[cfg.out_dtype]
    B, N, D, H, W, C = cfg.B, cfg.N, cfg.D, cfg.H, cfg.W, cfg.C
    X, Y, Z = cfg.X, cfg.Y, cfg.Z
    depth = np.empty((B, N, D, H, W), dtype=dt)
    feat = np.empty((B, N, H, W, C), dtype=dt)
    grad = np.empty((B, Z, Y, X, C), dtype=odt) if with_grad else None
    lg = np.empty((B, N, D, H, W), dtype=dt) if with_logits else None
    for b in range(B):
        logits = 3.0 * rng.standard_normal((N, D, H, W))
        depth[b] = _softmax_depth(logits).astype(dt)
        if with_logits:
            lg[b] = logits.astype(dt)
        feat[b] = rng.standard_normal((N, H, W, C)).astype(dt)
        if with_grad:
            grad[b] = rng.standard_normal((Z, Y, X, C)).astype(odt)
    out = {"depth": depth, "feat": feat, "grad_out": grad}
    if with_logits:
        out["logits"] = lg
    return out


def draw_small(rng: np.random.Generator, shape: dict, dtype: str = "f32",
               out_dtype: str | None = None, softmax: bool = True) -> dict:
    """Random activations for an arbitrary small shape (tests)."""
    dt = _NP_DTYPE[dtype]
    odt = _NP_DTYPE[out_dtype or dtype]
    B, N, D, H, W, C = (shape[k] for k in "BNDHWC")
    X, Y, Z = shape["X"], shape["Y"], shape["Z"]
    logits = 3.0 * rng.standard_normal((B, N, D, H, W))
    if softmax:
        depth = np.empty_like(logits)
        for b in range(B):
            depth[b] = _softmax_depth(logits[b])
    else:
        depth = rng.standard_normal((B, N, D, H, W))
    feat = rng.standard_normal((B, N, H, W, C))
    grad = rng.standard_normal((B, Z, Y, X, C))
    return {"depth": depth.astype(dt), "feat": feat.astype(dt),
            "grad_out": grad.astype(odt)}

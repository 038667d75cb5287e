"""Seeded synthetic boundary inputs for the GMC operator.

This module only draws random tensors; it contains none of the method's
arithmetic.  The same arrays feed the HIP path (through the C-ABI) and the
fp64 CPU oracle, so both see bit-identical inputs.

Every tensor is drawn with NumPy ``Generator(PCG64(seed))`` in float32.  For
bf16 workloads each value is rounded to the nearest bf16 (ties to even) on the
host; the rounded float32 array up-casts exactly to fp64 for the oracle and is
re-encoded as bf16 bits for the device.

Shapes follow the operator's boundary arguments (method section "Boundary
Message Geometry" and the appendix on native message clients):
  hidden  [B][N][d]          residual-stream visual states h_i
  text_q  [B][T][Hq][dh]     post-norm, post-rotary text queries
  vis_k   [B][N][Hkv][dh]    post-norm, post-rotary visual keys
  pos3d   [B][N][3] int32    original multimodal (t, h, w) position ids
  probe   [Hq][r][d]         folded value probe (W^V_kv(h) O_h P, per head)
  app_proj [app_rank][d]     +-1 Rademacher projection for the bounded
                             long-prefix appearance bank (only when needed)

Workload recipes (the paper's Qwen2.5-VL-7B and document settings stand in
as synthetic tensors of the same shape; no benchmark data is used):
  tiny    N=256 (16x16), T=16, d=512, 8/2 heads, dh=64, K=64, fp32, iid N(0,1)
  qwen    N=1296 (36x36), T=64, d=3584, 28/4 heads, dh=128, K=256, bf16,
          16-component Gaussian mixture, h = mu_z + 0.5 eps
  doc     N=4096 (64x64), T=128, K=820, bf16, 32 spatially contiguous
          (Voronoi) clusters, 5% outliers scaled 4x, queries aligned to 3
          clusters
  batch16 16 independent qwen problems in one call
  frames  N=16384 (4 frames of 64x64), T=256, K=2048, bf16, frame-to-frame
          correlation 0.9 of the within-cluster deviation; bounded bank
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "Problem", "make_problem", "round_bf16",
    "bf16_bits", "rademacher_projection", "APP_PROJ_SEED", "HistView", "make_history",
    "make_multi_image",
]

APP_PROJ_SEED = 104729  # seed of the long-prefix appearance projection


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    batch: int
    n: int
    grid_h: int
    grid_w: int
    frames: int
    t: int
    d: int
    hq: int
    hkv: int
    dh: int
    k: int
    dtype: str          # "f32" or "bf16"
    kind: str           # "iid", "mixture", "voronoi", "frames"
    n_centres: int = 16


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 256, 16, 16, 1, 16, 512, 8, 2, 64, 64, "f32", "iid"),
    "qwen": Workload("qwen", 1, 1, 1296, 36, 36, 1, 64, 3584, 28, 4, 128, 256, "bf16", "mixture"),
    "doc": Workload("doc", 2, 1, 4096, 64, 64, 1, 128, 3584, 28, 4, 128, 820, "bf16", "voronoi", 32),
    "batch16": Workload("batch16", 3, 16, 1296, 36, 36, 1, 64, 3584, 28, 4, 128, 256, "bf16", "mixture"),
    "frames": Workload("frames", 4, 1, 16384, 64, 64, 4, 256, 3584, 28, 4, 128, 2048, "bf16", "frames"),
}


@dataclasses.dataclass
class Problem:
    """One call's worth of inputs (float32 arrays holding the exact values)."""
    workload: Workload
    hidden: np.ndarray      # [B][N][d] float32
    text_q: np.ndarray      # [B][T][Hq][dh] float32
    vis_k: np.ndarray       # [B][N][Hkv][dh] float32
    pos3d: np.ndarray       # [B][N][3] int32
    probe: np.ndarray       # [Hq][r][d] float32
    app_proj: Optional[np.ndarray]  # [app_rank][d] float32 (+-1) or None
    k: int
    image_id: Optional[np.ndarray] = None   # [B][N] int32 for a multi-image prompt
    n_images: int = 1


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Bit patterns (uint16) of float32 values that are exactly bf16."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("array holds values that are not exactly bf16")
    return (u >> 16).astype(np.uint16)


def rademacher_projection(rank: int, d: int, seed: int = APP_PROJ_SEED) -> np.ndarray:
    """+-1 matrix [rank][d] from PCG64(seed); sign of a uniform 0/1 draw."""
    rng = np.random.Generator(np.random.PCG64(seed))
    bits = rng.integers(0, 2, size=(rank, d), dtype=np.int8)
    return (2.0 * bits - 1.0).astype(np.float32)


def _grid_positions(w: Workload) -> np.ndarray:
    """(t, h, w) ids, frame-major then row-major over the grid."""
    f, hh, ww = np.meshgrid(np.arange(w.frames), np.arange(w.grid_h),
                            np.arange(w.grid_w), indexing="ij")
    return np.stack([f.ravel(), hh.ravel(), ww.ravel()], axis=1).astype(np.int32)


def _normal(rng, shape, scale=1.0):
    return (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(scale))


def _mixture_states(rng, w: Workload, n_tokens: int):
    centres = _normal(rng, (w.n_centres, w.d))
    labels = rng.integers(0, w.n_centres, size=n_tokens)
    h = centres[labels] + _normal(rng, (n_tokens, w.d), 0.5)
    return h, centres, labels


def _voronoi_states(rng, w: Workload):
    n = w.n
    seeds = rng.choice(n, size=w.n_centres, replace=False)
    sy, sx = seeds // w.grid_w, seeds % w.grid_w
    yy, xx = np.divmod(np.arange(n), w.grid_w)
    dist = (yy[:, None] - sy[None, :]) ** 2 + (xx[:, None] - sx[None, :]) ** 2
    labels = np.argmin(dist, axis=1)            # first minimum: lower seed index
    centres = _normal(rng, (w.n_centres, w.d))
    h = centres[labels] + _normal(rng, (n, w.d), 0.5)
    n_out = int(round(0.05 * n))
    outliers = rng.choice(n, size=n_out, replace=False)
    h[outliers] *= np.float32(4.0)
    return h, labels


def _one_image(rng, w: Workload, wk: np.ndarray):
    """Draw one image's hidden/q/k; wk is the shared key map [d][Hkv*dh]."""
    if w.kind == "iid":
        h = _normal(rng, (w.n, w.d))
        q = _normal(rng, (w.t, w.hq, w.dh))
        k = _normal(rng, (w.n, w.hkv, w.dh))
        return h, q, k
    if w.kind == "mixture":
        h, _, _ = _mixture_states(rng, w, w.n)
        q = _normal(rng, (w.t, w.hq, w.dh))
    elif w.kind == "voronoi":
        h, labels = _voronoi_states(rng, w)
        keys = (h @ wk).reshape(w.n, w.hkv, w.dh)
        chosen = rng.choice(w.n_centres, size=3, replace=False)
        q = _normal(rng, (w.t, w.hq, w.dh))
        group = w.hq // w.hkv
        for t in range(w.t):
            c = chosen[t % 3]
            mk = keys[labels == c].mean(axis=0)                      # [Hkv][dh]
            mk = mk / np.linalg.norm(mk, axis=1, keepdims=True)
            for hh in range(w.hq):
                q[t, hh] += np.float32(3.0) * mk[hh // group]
    elif w.kind == "frames":
        per = w.grid_h * w.grid_w
        h0, centres, labels = _mixture_states(rng, w, per)
        frames = [h0]
        dev = h0 - centres[labels]
        for _ in range(1, w.frames):
            dev = np.float32(0.9) * dev + np.float32(np.sqrt(0.19)) * _normal(rng, (per, w.d), 0.5)
            frames.append(centres[labels] + dev)
        h = np.concatenate(frames, axis=0)
        q = _normal(rng, (w.t, w.hq, w.dh))
    else:
        raise ValueError(w.kind)
    k = (h @ wk).reshape(w.n, w.hkv, w.dh)
    return h, q, k


def make_problem(name: str, *, batch: Optional[int] = None, n: Optional[int] = None,
                 k: Optional[int] = None, t: Optional[int] = None,
                 grid: Optional[tuple] = None, seed: Optional[int] = None,
                 with_app_proj: Optional[bool] = None, app_rank: int = 128,
                 bounded_threshold: int = 4096) -> Problem:
    """Build the seeded inputs of a named workload.

    Keyword overrides shrink a workload (for parity tests at oracle-friendly
    sizes) while keeping its structure; ``grid`` = (frames, grid_h, grid_w).
    """
    w = WORKLOADS[name]
    repl = {}
    if grid is not None:
        repl.update(frames=grid[0], grid_h=grid[1], grid_w=grid[2],
                    n=grid[0] * grid[1] * grid[2])
    elif n is not None:
        raise ValueError("override n through grid=(frames, h, w)")
    if batch is not None:
        repl["batch"] = batch
    if k is not None:
        repl["k"] = k
    if t is not None:
        repl["t"] = t
    if seed is not None:
        repl["seed"] = seed
    if repl:
        w = dataclasses.replace(w, **repl)

    rng = np.random.Generator(np.random.PCG64(w.seed))
    probe = _normal(rng, (w.hq, 4, w.d), 1.0 / np.sqrt(w.d))
    wk = _normal(rng, (w.d, w.hkv * w.dh), 1.0 / np.sqrt(w.d))
    if w.batch == 1:
        streams = [rng]
    else:
        streams = [np.random.Generator(np.random.PCG64(s))
                   for s in np.random.SeedSequence(w.seed).spawn(w.batch)]
    hs, qs, ks = [], [], []
    for r in streams:
        h, q, kk = _one_image(r, w, wk)
        hs.append(h), qs.append(q), ks.append(kk)
    hidden = np.stack(hs).astype(np.float32)
    text_q = np.stack(qs).astype(np.float32)
    vis_k = np.stack(ks).astype(np.float32)
    if w.dtype == "bf16":
        hidden, text_q, vis_k = round_bf16(hidden), round_bf16(text_q), round_bf16(vis_k)
        probe = round_bf16(probe)
    pos = np.broadcast_to(_grid_positions(w), (w.batch, w.n, 3)).copy()
    if with_app_proj is None:
        with_app_proj = w.n > bounded_threshold
    app = rademacher_projection(app_rank, w.d) if with_app_proj else None
    return Problem(w, np.ascontiguousarray(hidden), np.ascontiguousarray(text_q),
                   np.ascontiguousarray(vis_k), pos, np.ascontiguousarray(probe), app, w.k)


@dataclasses.dataclass
class HistView:
    """One completed historical message view of a problem (the residual
    states entering an earlier block, that block's queries and keys, and its
    folded value probe)."""
    hidden: np.ndarray      # [B][N][d] float32
    text_q: np.ndarray      # [B][T][Hq][dh] float32
    vis_k: np.ndarray       # [B][N][Hkv][dh] float32
    probe: np.ndarray       # [Hq][r][d] float32


def make_history(prob: Problem, n_views: int = 2) -> list:
    """Historical views of a problem, view v drawn from its own stream
    (SeedSequence(seed).spawn(...) children past the batch's): states one and
    two blocks earlier differ from the boundary's by a residual update,
    h_v = h - 0.25 (v + 1) eps; queries keep most of the boundary queries,
    q_v = 0.8 q + 0.6 eps; keys come from the view's states through the
    view's own key map W_K,v ~ N(0, 1/d); the folded probe G_v ~ N(0, 1/d).
    bf16 workloads are rounded like the boundary tensors."""
    w = prob.workload
    kids = np.random.SeedSequence(w.seed).spawn(w.batch + n_views)[w.batch:]
    views = []
    for v in range(n_views):
        rng = np.random.Generator(np.random.PCG64(kids[v]))
        probe = _normal(rng, (w.hq, prob.probe.shape[1], w.d), 1.0 / np.sqrt(w.d))
        wk = _normal(rng, (w.d, w.hkv * w.dh), 1.0 / np.sqrt(w.d))
        h = prob.hidden - _normal(rng, prob.hidden.shape, 0.25 * (v + 1))
        q = np.float32(0.8) * prob.text_q + _normal(rng, prob.text_q.shape, 0.6)
        k = np.einsum("bnd,de->bne", h, wk).reshape(w.batch, w.n, w.hkv, w.dh).astype(np.float32)
        if w.dtype == "bf16":
            h, q, k, probe = round_bf16(h), round_bf16(q), round_bf16(k), round_bf16(probe)
        views.append(HistView(np.ascontiguousarray(h, np.float32), np.ascontiguousarray(q, np.float32),
                              np.ascontiguousarray(k, np.float32), np.ascontiguousarray(probe, np.float32)))
    return views


def make_multi_image(name: str, grids, *, t: Optional[int] = None, k: Optional[int] = None,
                     seed: Optional[int] = None, batch: int = 1) -> Problem:
    """A multi-image prompt: the images' visual tokens one after another,
    image g on its own (grid_h, grid_w) grid with positions (g, row, col),
    each image's states an independent draw of the workload's state model
    (its own mixture centres), keys through the shared key map; queries over
    all images.  Images are drawn from SeedSequence children of the seed, one
    per (problem, image)."""
    w0 = WORKLOADS[name]
    n = int(sum(gh * gw for gh, gw in grids))
    repl = dict(batch=batch, n=n, frames=1, grid_h=0, grid_w=0)
    if t is not None:
        repl["t"] = t
    if k is not None:
        repl["k"] = k
    if seed is not None:
        repl["seed"] = seed
    w = dataclasses.replace(w0, **repl)
    rng = np.random.Generator(np.random.PCG64(w.seed))
    probe = _normal(rng, (w.hq, 4, w.d), 1.0 / np.sqrt(w.d))
    wk = _normal(rng, (w.d, w.hkv * w.dh), 1.0 / np.sqrt(w.d))
    kids = np.random.SeedSequence(w.seed).spawn(batch * (len(grids) + 1))
    hs, qs, ks, ps, ids = [], [], [], [], []
    for b in range(batch):
        hb, pb, ib = [], [], []
        for g, (gh, gw) in enumerate(grids):
            r = np.random.Generator(np.random.PCG64(kids[b * (len(grids) + 1) + g]))
            wg = dataclasses.replace(w, n=gh * gw, grid_h=gh, grid_w=gw, frames=1)
            h, _, _ = (_mixture_states(r, wg, gh * gw) if w.kind != "iid" else (_normal(r, (gh * gw, w.d)), 0, 0))
            hb.append(h)
            yy, xx = np.divmod(np.arange(gh * gw), gw)
            pb.append(np.stack([np.full(gh * gw, g), yy, xx], axis=1))
            ib.append(np.full(gh * gw, g))
        h = np.concatenate(hb, axis=0)
        rq = np.random.Generator(np.random.PCG64(kids[b * (len(grids) + 1) + len(grids)]))
        hs.append(h)
        qs.append(_normal(rq, (w.t, w.hq, w.dh)))
        ks.append((h @ wk).reshape(n, w.hkv, w.dh))
        ps.append(np.concatenate(pb, axis=0))
        ids.append(np.concatenate(ib))
    hidden = np.stack(hs).astype(np.float32)
    text_q = np.stack(qs).astype(np.float32)
    vis_k = np.stack(ks).astype(np.float32)
    if w.dtype == "bf16":
        hidden, text_q, vis_k = round_bf16(hidden), round_bf16(text_q), round_bf16(vis_k)
        probe = round_bf16(probe)
    return Problem(w, np.ascontiguousarray(hidden), np.ascontiguousarray(text_q), np.ascontiguousarray(vis_k),
                   np.stack(ps).astype(np.int32), np.ascontiguousarray(probe), None, w.k,
                   np.stack(ids).astype(np.int32), len(grids))

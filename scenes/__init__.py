"""Seeded synthetic multi-view token scenes.

A scene is what a visual-geometric encoder hands to a token pruner: N visual
tokens, each with a feature embedding, a 3D world position and the index of
the frame it came from, plus a per-token target capacity and a budget K
(problem setup, Sec. 3.2 of the paper).  The paper's workloads are 32-frame
indoor videos run through 3D VLM encoders; neither the videos nor the
encoders are available, so these scenes stand in for them with the same
shapes and structure: objects that recur across frames, multi-view position
noise along camera rays, and a fraction of outlier tokens.

This module is shared by the GPU library's tests and benchmark and by the CPU
oracle.  It holds none of the method's arithmetic: it only draws tokens and
assigns capacities by two plain recipes (uniform, or proportional to the
token count of the token's object).

Storage: positions float32 [N,3] metres, frames int32 [N], capacities
float32 [N] summing to 1 (up to float32 rounding).  Features are float32
[N,D], or bfloat16 stored as uint16 bit patterns [N,D] rounded once from
float32 with round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

__all__ = ["SceneConfig", "Scene", "CONFIGS", "make_scene", "f32_to_bf16_bits", "to_device",
           "bf16_bits_to_f32", "subscene"]


@dataclass(frozen=True)
class SceneConfig:
    name: str
    n_frames: int
    per_frame: int
    dim: int
    dtype: str                      # "f32" or "bf16"
    k: int                          # budget
    n_objects: int
    zipf: Optional[float]           # object weight exponent; None = uniform
    box_lo: Tuple[float, float, float]
    box_hi: Tuple[float, float, float]
    outlier_frac: float
    capacity: str                   # "uniform" | "density"
    orbit: bool                     # positions get depth noise along camera rays
    views: Optional[Tuple[int, int]]  # frames each object is visible in (min, max)
    jitter: float                   # per-(object, frame) feature jitter scale
    noise: float = 0.3              # per-token feature noise scale
    sigma_obj: float = 0.25         # object spread per axis, metres
    depth_sigma: float = 0.05       # depth noise along the camera ray, metres
    orbit_radius: float = 3.0
    camera_height: float = 1.5
    voxel: Optional[float] = None   # Lite voxel size, metres
    path: str = "full"              # "full" (cost + greedy) or "lite"
    # The workload's capacities come from the FST capacity of Eq. 9-10 with
    # this many 3D neighbours per token (None: the generator's own recipe
    # above is the workload's).  The generator does not compute it: that is
    # the method's arithmetic, done by the library for the benchmark and by
    # the oracle for the parity tests; `capacity` stays the generator's
    # recipe for every other use of the scene.
    fst_capacity_nn: Optional[int] = None

    @property
    def n(self) -> int:
        return self.n_frames * self.per_frame


# The five workloads the path is measured and checked on, named by what they
# are.  Box extents not fixed by the workload description are chosen so that
# the 3 m camera orbit encloses the objects.  Capacities: uniform for the
# 8192-token scene, proportional to the token count of the token's object for
# the 16384-token room, and the FST capacity (8 or 16 neighbours) for the
# other three.
CONFIGS = {
    # 1024 tokens (8 frames x 128), 256-d float32 features, K = 102 (10 %).
    "n1024_d256_f32": SceneConfig(
        "n1024_d256_f32", 8, 128, 256, "f32", 102, 12, None,
        (0.0, 0.0, 0.0), (6.0, 6.0, 3.0), 0.05, "density", False, None, 0.0, fst_capacity_nn=8),
    # 4096 tokens (16 frames x 16x16 patches), 1152-d bf16, K = 410 (10 %).
    "n4096_d1152": SceneConfig(
        "n4096_d1152", 16, 256, 1152, "bf16", 410, 40, 1.2,
        (-2.0, -2.0, 0.0), (2.0, 2.0, 2.5), 0.05, "density", True, None, 0.0, fst_capacity_nn=16),
    # 8192 tokens (32 frames x 256), 3584-d bf16 (LLM width), K = 1229 (15 %).
    "n8192_d3584": SceneConfig(
        "n8192_d3584", 32, 256, 3584, "bf16", 1229, 80, 1.2,
        (-2.5, -2.5, 0.0), (2.5, 2.5, 3.0), 0.05, "uniform", True, (4, 12), 0.2),
    # 16384 tokens (64 frames x 256), 3584-d bf16, K = 1638 (10 %), 10x10x3 m room.
    "n16384_d3584": SceneConfig(
        "n16384_d3584", 64, 256, 3584, "bf16", 1638, 160, 1.1,
        (-5.0, -5.0, 0.0), (5.0, 5.0, 3.0), 0.08, "density", True, (4, 12), 0.2),
    # Lite: 32768 tokens (128 frames x 256), 3584-d bf16, K = 3277, 0.25 m voxels.
    "lite_n32768_d3584": SceneConfig(
        "lite_n32768_d3584", 128, 256, 3584, "bf16", 3277, 300, 1.2,
        (-8.0, -8.0, 0.0), (8.0, 8.0, 3.0), 0.05, "uniform", True, (4, 12), 0.2,
        voxel=0.25, path="lite", fst_capacity_nn=16),
    # The paper's own efficiency shape: 32 frames x 196 tokens = 6272 -> 628.
    "paper_n6272_d3584": SceneConfig(
        "paper_n6272_d3584", 32, 196, 3584, "bf16", 628, 80, 1.2,
        (-2.5, -2.5, 0.0), (2.5, 2.5, 3.0), 0.05, "uniform", True, (4, 12), 0.2,
        voxel=0.25),
}


@dataclass
class Scene:
    config: SceneConfig
    seed: int
    feats: np.ndarray       # float32 [N,D] or uint16 bf16 bits [N,D]
    dtype: str              # "f32" | "bf16"
    pos: np.ndarray         # float32 [N,3]
    frame: np.ndarray       # int32 [N]
    capacity: np.ndarray    # float32 [N]
    k: int
    obj: np.ndarray         # int32 [N], -1 for outliers

    @property
    def n(self) -> int:
        return int(self.pos.shape[0])

    @property
    def dim(self) -> int:
        return int(self.feats.shape[1])

    def feats_f32(self) -> np.ndarray:
        if self.dtype == "bf16":
            return bf16_bits_to_f32(self.feats)
        return self.feats


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normalise_rows(a: np.ndarray) -> np.ndarray:
    a64 = a.astype(np.float64)
    nrm = np.sqrt(np.einsum("ij,ij->i", a64, a64))
    nrm[nrm == 0] = 1.0
    return (a64 / nrm[:, None]).astype(np.float32)


def make_scene(config, seed: int = 0, **overrides) -> Scene:
    """Draw one scene.  ``config`` is a SceneConfig or a key of CONFIGS;
    keyword overrides replace config fields (e.g. a smaller frame count for a
    quick parity case).

    Draw order (one PCG64 stream): object prototypes, centres, cameras,
    visibility, outlier slots, token-to-object choice, per-visit jitter,
    token feature noise, position noise, depth noise, outlier features and
    positions.
    """
    cfg = CONFIGS[config] if isinstance(config, str) else config
    if overrides:
        cfg = dataclasses.replace(cfg, **overrides)
    rng = np.random.default_rng(seed)
    n, d, n_obj, n_fr, per = cfg.n, cfg.dim, cfg.n_objects, cfg.n_frames, cfg.per_frame
    lo = np.asarray(cfg.box_lo, np.float64)
    hi = np.asarray(cfg.box_hi, np.float64)

    protos = rng.standard_normal((n_obj, d), dtype=np.float32)
    centres = rng.uniform(lo, hi, size=(n_obj, 3))
    if cfg.zipf is None:
        w = np.ones(n_obj)
    else:
        w = np.arange(1, n_obj + 1, dtype=np.float64) ** (-cfg.zipf)
    w = w / w.sum()

    if cfg.orbit:
        theta = rng.uniform(0.0, 2.0 * math.pi, size=n_fr)
        cx, cy = 0.5 * (lo[0] + hi[0]), 0.5 * (lo[1] + hi[1])
        cams = np.stack([cx + cfg.orbit_radius * np.cos(theta),
                         cy + cfg.orbit_radius * np.sin(theta),
                         np.full(n_fr, cfg.camera_height)], axis=1)
    else:
        cams = None

    visible = [list(range(n_obj)) for _ in range(n_fr)]
    if cfg.views is not None:
        sets = [[] for _ in range(n_fr)]
        vmin, vmax = cfg.views
        for k in range(n_obj):
            nv = min(int(rng.integers(vmin, vmax + 1)), n_fr)
            for f in rng.choice(n_fr, size=nv, replace=False):
                sets[int(f)].append(k)
        visible = [sorted(s) if s else list(range(n_obj)) for s in sets]

    n_out = int(round(cfg.outlier_frac * n))
    out_slots = np.sort(rng.choice(n, size=n_out, replace=False)) if n_out else np.zeros(0, np.int64)
    is_out = np.zeros(n, bool)
    is_out[out_slots] = True

    frame = (np.arange(n) // per).astype(np.int32)
    obj = np.full(n, -1, np.int32)
    for f in range(n_fr):
        slots = np.nonzero(~is_out[f * per:(f + 1) * per])[0] + f * per
        vis = np.asarray(visible[f])
        p = w[vis] / w[vis].sum()
        obj[slots] = rng.choice(vis, size=slots.size, p=p)

    visit_row = {}
    if cfg.jitter > 0:
        for f in range(n_fr):
            for k in visible[f]:
                visit_row[(f, k)] = len(visit_row)
        jit = rng.standard_normal((len(visit_row), d), dtype=np.float32)

    eps = rng.standard_normal((n, d), dtype=np.float32)
    feats = np.empty((n, d), np.float32)
    inl = ~is_out
    feats[inl] = protos[obj[inl]] + np.float32(cfg.noise) * eps[inl]
    if cfg.jitter > 0:
        rows = np.nonzero(inl)[0]
        vr = np.fromiter((visit_row[(int(frame[i]), int(obj[i]))] for i in rows),
                         dtype=np.int64, count=rows.size)
        feats[rows] += np.float32(cfg.jitter) * jit[vr]
        del jit
    del eps

    pos = np.zeros((n, 3), np.float64)
    pos[inl] = centres[obj[inl]] + cfg.sigma_obj * rng.standard_normal((int(inl.sum()), 3))
    if cams is not None:
        o = cams[frame[inl]]
        ray = pos[inl] - o
        r = np.linalg.norm(ray, axis=1)
        r = np.where(r > 0, r, 1.0)
        depth = r + cfg.depth_sigma * rng.standard_normal(r.shape[0])
        pos[inl] = o + (depth / r)[:, None] * ray

    if n_out:
        feats[out_slots] = rng.standard_normal((n_out, d), dtype=np.float32)
        pos[out_slots] = rng.uniform(lo, hi, size=(n_out, 3))

    feats = _normalise_rows(feats)

    if cfg.capacity == "uniform":
        cap = np.full(n, 1.0 / n)
    elif cfg.capacity == "density":
        counts = np.bincount(obj[inl], minlength=n_obj).astype(np.float64)
        cap = np.where(inl, counts[np.maximum(obj, 0)], 1.0)
        cap = cap / cap.sum()
    else:
        raise ValueError(f"unknown capacity recipe {cfg.capacity!r}")

    if cfg.dtype == "bf16":
        feats_out = f32_to_bf16_bits(feats)
    elif cfg.dtype == "f32":
        feats_out = feats
    else:
        raise ValueError(f"unknown feature dtype {cfg.dtype!r}")
    return Scene(cfg, seed, np.ascontiguousarray(feats_out), cfg.dtype,
                 pos.astype(np.float32), frame, cap.astype(np.float32),
                 int(cfg.k), obj)


def subscene(scene: Scene, idx, k: Optional[int] = None, renormalise: bool = True) -> Scene:
    """Tokens ``idx`` of a scene, with capacities renormalised to sum 1."""
    idx = np.asarray(idx)
    cap = scene.capacity[idx].astype(np.float64)
    if renormalise and cap.sum() > 0:
        cap = cap / cap.sum()
    return Scene(scene.config, scene.seed, np.ascontiguousarray(scene.feats[idx]), scene.dtype,
                 np.ascontiguousarray(scene.pos[idx]), np.ascontiguousarray(scene.frame[idx]),
                 cap.astype(np.float32), scene.k if k is None else int(k),
                 np.ascontiguousarray(scene.obj[idx]))


def to_device(scene: Scene, device="cuda"):
    """The scene's arrays as torch tensors on ``device`` (features as
    torch.bfloat16 or torch.float32).  Plain data movement."""
    import torch
    if scene.dtype == "bf16":
        feats = torch.from_numpy(scene.feats.view(np.int16)).view(torch.bfloat16)
    else:
        feats = torch.from_numpy(scene.feats)
    return dict(
        feats=feats.to(device).contiguous(),
        pos=torch.from_numpy(scene.pos).to(device).contiguous(),
        frame=torch.from_numpy(scene.frame).to(device).contiguous(),
        capacity=torch.from_numpy(scene.capacity).to(device).contiguous(),
    )

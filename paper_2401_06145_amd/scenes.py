"""Seeded synthetic point-cloud scenes that stand in for the paper's datasets.

The paper evaluates on voxelised real scans (outdoor LiDAR, indoor scans) and on
uniform random clouds (Section 6.1, Datasets).  None of those datasets is
available here, so every workload is generated from a fixed seed with the same
structure: unique integer voxel coordinates (b, x, y, z), an N x C feature matrix
and per-offset weights W[k][C_in][C_out].

This module is the ONLY code shared by the CPU oracle's tests and the GPU path's
tests.  It holds no arithmetic of the sparse-convolution method itself: it only
draws points, voxelises them (floor of point / voxel size), removes duplicate
voxels, shuffles rows and draws feature / weight values.

Random streams (numpy PCG64): geometry ``1000 + i``, features ``2000 + i``,
weights ``3000 + i`` for scene recipe ``i``.  Values are drawn in float64 and
rounded to the requested dtype (round-to-nearest-even).  Rows are always returned
in a seeded random order so that unsorted input is exercised.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

# Point budgets, calibrated once so that the unique-voxel count lands within +-3%
# of the recipe's target (the test suite re-checks the counts).
LIDAR_BUDGET_120K = 298_000
LIDAR_BUDGET_200K = 545_000
INDOOR_BUDGET_300K = 355_000


def _round_to(a: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> dtype with round-to-nearest-even, returned as that dtype."""
    if dtype == "f32":
        return a.astype(np.float32)
    if dtype == "f16":
        return a.astype(np.float16)
    if dtype == "bf16":
        # RNE to bfloat16, stored as uint16 bit patterns (numpy has no bf16).
        f = a.astype(np.float32).view(np.uint32).astype(np.uint64)
        lsb = (f >> 16) & 1
        r = ((f + 0x7FFF + lsb) >> 16).astype(np.uint16)
        return r
    raise ValueError(dtype)


def bf16_bits_to_f64(u: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float64."""
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a feature / weight array in ``dtype`` to float64."""
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    return a.astype(np.float64)


def features(n: int, c: int, dtype: str, seed: int) -> np.ndarray:
    """N(0,1) features [n][c] drawn in float64, rounded to dtype."""
    rng = np.random.default_rng(seed)
    return _round_to(rng.standard_normal((n, c)), dtype)


def weights(K: int, c_in: int, c_out: int, dtype: str, seed: int) -> np.ndarray:
    """W[k][c_in][c_out] ~ N(0, 1/(K^3 c_in)), rounded to dtype."""
    rng = np.random.default_rng(seed)
    k3 = K ** 3
    std = 1.0 / np.sqrt(k3 * c_in)
    return _round_to(rng.standard_normal((k3, c_in, c_out)) * std, dtype)


def _finish(coords: np.ndarray, rng: np.random.Generator) -> np.ndarray:
    """Deduplicate voxels and return them, int32 [n][4], in a seeded random row order."""
    u = np.unique(coords, axis=0)
    perm = rng.permutation(u.shape[0])
    return np.ascontiguousarray(u[perm].astype(np.int32))


def coords_sha256(coords: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(coords, dtype=np.int32).tobytes()).hexdigest()


# ----------------------------------------------------------------------------
# Uniform random cells (the paper's "Random" set, Section 6.1)
# ----------------------------------------------------------------------------

def uniform_cells(n: int, side: int, seed: int, batch: int = 0) -> np.ndarray:
    """``n`` distinct cells drawn without replacement from a side^3 grid (b = batch)."""
    rng = np.random.default_rng(seed)
    cells = rng.choice(side ** 3, n, replace=False)
    x = cells // (side * side)
    y = (cells // side) % side
    z = cells % side
    b = np.full(n, batch, dtype=np.int64)
    c = np.stack([b, x, y, z], axis=1).astype(np.int32)
    # rng.choice order is already random; keep it (unique by construction).
    return np.ascontiguousarray(c)


def uniform_cells_large(n: int, side: int, seed: int, batch: int = 0) -> np.ndarray:
    """``n`` distinct cells of a side^3 grid for large n (draws with replacement,
    keeps distinct cells, trims to n in a seeded random order)."""
    rng = np.random.default_rng(seed)
    total = side ** 3
    if n > total // 2:
        raise ValueError("density too high for rejection drawing")
    cells = np.unique(rng.integers(0, total, int(n * 1.1) + 1024, dtype=np.int64))
    while cells.size < n:
        cells = np.unique(np.concatenate([cells, rng.integers(0, total, n, dtype=np.int64)]))
    cells = cells[rng.permutation(cells.size)[:n]]
    x = cells // (side * side)
    y = (cells // side) % side
    z = cells % side
    b = np.full(n, batch, dtype=np.int64)
    return np.ascontiguousarray(np.stack([b, x, y, z], axis=1).astype(np.int32))


# ----------------------------------------------------------------------------
# LiDAR-like outdoor scene
# ----------------------------------------------------------------------------

def _sample_box_surface(rng, n, cx, cy, wx, wy, h):
    """n points uniformly on the 4 side faces + top face of an axis-aligned box on z=0."""
    areas = np.array([wx * h, wx * h, wy * h, wy * h, wx * wy])
    face = rng.choice(5, n, p=areas / areas.sum())
    u = rng.random(n)
    v = rng.random(n)
    x = np.empty(n)
    y = np.empty(n)
    z = np.empty(n)
    x0, y0 = cx - wx / 2, cy - wy / 2
    # faces 0/1: y = y0 / y0+wy ; faces 2/3: x = x0 / x0+wx ; face 4: top
    m = face == 0
    x[m], y[m], z[m] = x0 + u[m] * wx, y0, v[m] * h
    m = face == 1
    x[m], y[m], z[m] = x0 + u[m] * wx, y0 + wy, v[m] * h
    m = face == 2
    x[m], y[m], z[m] = x0, y0 + u[m] * wy, v[m] * h
    m = face == 3
    x[m], y[m], z[m] = x0 + wx, y0 + u[m] * wy, v[m] * h
    m = face == 4
    x[m], y[m], z[m] = x0 + u[m] * wx, y0 + v[m] * wy, h
    return x, y, z


def _sample_cylinder_surface(rng, n, cx, cy, r, h):
    """n points uniformly on the lateral surface + top disk of a vertical cylinder."""
    areas = np.array([2 * np.pi * r * h, np.pi * r * r])
    part = rng.choice(2, n, p=areas / areas.sum())
    th = rng.random(n) * 2 * np.pi
    x = np.empty(n)
    y = np.empty(n)
    z = np.empty(n)
    m = part == 0
    x[m], y[m], z[m] = cx + r * np.cos(th[m]), cy + r * np.sin(th[m]), rng.random(m.sum()) * h
    m = part == 1
    rr = r * np.sqrt(rng.random(m.sum()))
    x[m], y[m], z[m] = cx + rr * np.cos(th[m]), cy + rr * np.sin(th[m]), h
    return x, y, z


def lidar_points(seed: int, budget: int) -> np.ndarray:
    """Raw float points [n][3] of one LiDAR-like scene (metres)."""
    rng = np.random.default_rng(seed)
    n_ground = budget // 2
    n_obj = budget - n_ground
    # Ground z = 0: radius log-uniform in [2, 70.7] m => areal density ~ 1/r^2.
    r = np.exp(rng.uniform(np.log(2.0), np.log(70.7), n_ground))
    th = rng.uniform(0, 2 * np.pi, n_ground)
    gx, gy = r * np.cos(th), r * np.sin(th)
    keep = (np.abs(gx) < 50) & (np.abs(gy) < 50)
    pts = [np.stack([gx[keep], gy[keep], np.zeros(keep.sum())], axis=1)]
    # 40 objects: 20 boxes, 20 vertical cylinders, centres in [-45,45]^2 and >= 3 m from origin.
    centres = []
    while len(centres) < 40:
        c = rng.uniform(-45, 45, 2)
        if np.hypot(c[0], c[1]) >= 3.0:
            centres.append(c)
    shapes = []
    for i in range(40):
        cx, cy = centres[i]
        if i < 20:
            wx, wy, h = rng.uniform(1, 8), rng.uniform(1, 8), rng.uniform(1, 6)
            shapes.append(("box", cx, cy, wx, wy, h, 2 * (wx + wy) * h + wx * wy))
        else:
            rad, h = rng.uniform(0.1, 1.0), rng.uniform(1, 8)
            shapes.append(("cyl", cx, cy, rad, h, 0.0, 2 * np.pi * rad * h + np.pi * rad * rad))
    area = np.array([s[-1] for s in shapes])
    per = rng.multinomial(n_obj, area / area.sum())
    for s, n in zip(shapes, per):
        if n == 0:
            continue
        if s[0] == "box":
            x, y, z = _sample_box_surface(rng, n, s[1], s[2], s[3], s[4], s[5])
        else:
            x, y, z = _sample_cylinder_surface(rng, n, s[1], s[2], s[3], s[4])
        rh = np.hypot(x, y)
        acc = np.minimum(1.0, (5.0 / np.maximum(rh, 1e-9)) ** 2)
        keep = rng.random(n) < acc
        pts.append(np.stack([x[keep], y[keep], z[keep]], axis=1))
    p = np.concatenate(pts, axis=0)
    p[:, 0] = np.clip(p[:, 0], -50.0, np.nextafter(50.0, 0))
    p[:, 1] = np.clip(p[:, 1], -50.0, np.nextafter(50.0, 0))
    p[:, 2] = np.clip(p[:, 2], 0.0, np.nextafter(8.0, 0))
    return p


def voxelise(points: np.ndarray, voxel: float, batch: int = 0) -> np.ndarray:
    """floor(point / voxel) -> int64 [n][4] with the batch index first (duplicates kept)."""
    q = np.floor(points / voxel).astype(np.int64)
    b = np.full((q.shape[0], 1), batch, dtype=np.int64)
    return np.concatenate([b, q], axis=1)


def lidar_scene(seed: int, budget: int = LIDAR_BUDGET_120K, batch: int = 0) -> np.ndarray:
    """Unique LiDAR-like voxels at 5 cm: x,y in [-1000, 999], z in [0, 159]."""
    v = voxelise(lidar_points(seed, budget), 0.05, batch)
    return _finish(v, np.random.default_rng(seed + 7919))


def lidar_batch(n_target: int, seed: int, distinct: int = 8) -> np.ndarray:
    """A batch of LiDAR-like frames of about ``n_target`` voxels in all: whole frames
    of ~120k voxels, frame f at batch index f.  The first ``distinct`` frames have
    their own geometry (seeds seed + f); later frames repeat those geometries under
    new batch indices.  Rows in a seeded random order."""
    frames = max(1, -(-n_target // 120_357))
    geo = [lidar_scene(seed + f, LIDAR_BUDGET_120K, batch=0) for f in range(min(frames, distinct))]
    parts = []
    for f in range(frames):
        g = geo[f % len(geo)].copy()
        g[:, 0] = f
        parts.append(g)
    c = np.concatenate(parts, axis=0)
    rng = np.random.default_rng(seed + 104729)
    return np.ascontiguousarray(c[rng.permutation(c.shape[0])])


# ----------------------------------------------------------------------------
# Indoor-like room
# ----------------------------------------------------------------------------

def indoor_points(seed: int, budget: int) -> np.ndarray:
    """Raw float points of a 10 x 8 x 3 m room (floor, ceiling, 4 walls) with 30 boxes."""
    rng = np.random.default_rng(seed)
    L, W, H = 10.0, 8.0, 3.0
    # planar patches: (origin, edge u, edge v)
    patches = [
        (np.array([0, 0, 0.0]), np.array([L, 0, 0.0]), np.array([0, W, 0.0])),  # floor
        (np.array([0, 0, H]), np.array([L, 0, 0.0]), np.array([0, W, 0.0])),  # ceiling
        (np.array([0, 0, 0.0]), np.array([L, 0, 0.0]), np.array([0, 0, H])),  # wall y=0
        (np.array([0, W, 0.0]), np.array([L, 0, 0.0]), np.array([0, 0, H])),  # wall y=W
        (np.array([0, 0, 0.0]), np.array([0, W, 0.0]), np.array([0, 0, H])),  # wall x=0
        (np.array([L, 0, 0.0]), np.array([0, W, 0.0]), np.array([0, 0, H])),  # wall x=L
    ]
    for _ in range(30):
        wx, wy, h = rng.uniform(0.3, 2.0), rng.uniform(0.3, 2.0), rng.uniform(0.3, 2.0)
        x0 = rng.uniform(0, L - wx)
        y0 = rng.uniform(0, W - wy)
        o = np.array([x0, y0, 0.0])
        ex, ey, ez = np.array([wx, 0, 0.0]), np.array([0, wy, 0.0]), np.array([0, 0, h])
        patches += [
            (o, ex, ez), (o + ey, ex, ez), (o, ey, ez), (o + ex, ey, ez), (o + ez, ex, ey),
        ]
    area = np.array([np.linalg.norm(np.cross(u, v)) for _, u, v in patches])
    per = rng.multinomial(budget, area / area.sum())
    pts = []
    for (o, u, v), n in zip(patches, per):
        a = rng.random((n, 1))
        b = rng.random((n, 1))
        pts.append(o + a * u + b * v)
    p = np.concatenate(pts, axis=0)
    p[:, 0] = np.clip(p[:, 0], 0.0, np.nextafter(L, 0))
    p[:, 1] = np.clip(p[:, 1], 0.0, np.nextafter(W, 0))
    p[:, 2] = np.clip(p[:, 2], 0.0, np.nextafter(H, 0))
    return p


def indoor_scene(seed: int, budget: int = INDOOR_BUDGET_300K, batch: int = 0) -> np.ndarray:
    """Unique indoor voxels at 2 cm: grid 500 x 400 x 150."""
    v = voxelise(indoor_points(seed, budget), 0.02, batch)
    return _finish(v, np.random.default_rng(seed + 7919))


# ----------------------------------------------------------------------------
# The five workloads
# ----------------------------------------------------------------------------

@dataclass
class Layer:
    """One sparse-conv layer of a workload: kernel size, stride, mode, channels, dtype."""
    K: int
    stride: int
    mode: str  # "subm" | "down" | "up"
    c_in: int
    c_out: int
    dtype: str
    tensor_stride: int = 1


@dataclass
class Workload:
    name: str
    coords: np.ndarray  # int32 [n][4]
    layers: list = field(default_factory=list)
    seed: int = 0


def workload(i: int, c: int | None = None) -> Workload:
    """Scene and layer recipe ``i`` (0..4).  ``c`` picks the channel width of recipe 3."""
    gs, fs = 1000 + i, 2000 + i
    if i == 0:
        coords = uniform_cells(2000, 64, gs)
        return Workload("uniform-2k-64cube-subm-k3-c16-f32", coords,
                        [Layer(3, 1, "subm", 16, 16, "f32")], i)
    if i == 1:
        coords = lidar_scene(gs, LIDAR_BUDGET_120K)
        return Workload("lidar-120k-subm-k3-c64-f16", coords,
                        [Layer(3, 1, "subm", 64, 64, "f16")], i)
    if i == 2:
        coords = lidar_scene(gs, LIDAR_BUDGET_200K)
        return Workload("lidar-200k-down-k2s2-c32to64-up-c64to32-f16", coords,
                        [Layer(2, 2, "down", 32, 64, "f16"), Layer(2, 2, "up", 64, 32, "f16")], i)
    if i == 3:
        cc = 64 if c is None else c
        coords = indoor_scene(gs, INDOOR_BUDGET_300K)
        return Workload(f"indoor-300k-subm-k3-c{cc}-f16", coords,
                        [Layer(3, 1, "subm", cc, cc, "f16")], i)
    if i == 4:
        a = lidar_scene(1004, LIDAR_BUDGET_120K, batch=0)
        b = lidar_scene(1104, LIDAR_BUDGET_120K, batch=1)
        rng = np.random.default_rng(gs + 7919)
        both = np.concatenate([a, b], axis=0)
        coords = np.ascontiguousarray(both[rng.permutation(both.shape[0])])
        return Workload("unet-2x-lidar-240k-f16", coords, [], i)
    raise ValueError(i)

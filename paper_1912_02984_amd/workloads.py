"""Seeded synthetic point-cloud workloads for the CAGQ hot path.

This module only draws inputs. It holds none of CAGQ's own arithmetic
(voxelization, tables, sampling, querying): both the HIP path and the CPU
oracle receive the same float32 arrays from here and nothing else.

The paper evaluates CAGQ on ModelNet40 objects and ScanNet / S3DIS rooms
(Sec. 4 and 5, Table "tab:query", Table "tb:morecond"), none of which are
available offline. The generators below stand in for them with the shapes,
sizes and density structure of those workloads:

* ``tiny``   - uniform points in the unit cube (a parity-only case);
* ``object`` - ModelNet-like objects: surfaces of 1-4 random primitives,
  normalised to the unit sphere, Gaussian noise;
* ``room``   - ScanNet-like indoor scenes: floor, four walls and random
  axis-aligned boxes, density thinned by distance to a sensor;
* ``lidar``  - a 64-ring spinning sensor sweep over a ground plane and boxes.

Every generator is a pure function of its seed (numpy ``default_rng``).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

__all__ = [
    "GridSpec", "LayerSpec", "Workload", "WORKLOADS", "get_workload",
    "uniform_cube", "object_clouds", "room_scenes", "lidar_sweep",
]


@dataclasses.dataclass(frozen=True)
class GridSpec:
    """Voxel grid: origin, per-axis voxel size, dims, cap n_v and radius r."""
    origin: Tuple[float, float, float]
    voxel_size: Tuple[float, float, float]
    dims: Tuple[int, int, int]
    n_v: int
    radius: int


@dataclasses.dataclass(frozen=True)
class LayerSpec:
    """One CAGQ layer: grid, M centers by 'rvs'/'cas', K nodes by 'cube'/'knn'."""
    grid: GridSpec
    M: int
    K: int
    sample: str
    query: str
    seed: int


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    layers: Tuple[LayerSpec, ...]
    data_seed: int
    description: str

    def points(self, B: Optional[int] = None) -> np.ndarray:
        """float32 [B, N, 3] for this workload (B defaults to self.B)."""
        b = self.B if B is None else B
        return _GENERATORS[self.name.split("/")[0]](b, self.N, self.data_seed)


# ---------------------------------------------------------------------------
# generators
# ---------------------------------------------------------------------------

def uniform_cube(B: int, N: int, seed: int) -> np.ndarray:
    """i.i.d. uniform points in [0, 1)^3."""
    rng = np.random.default_rng(seed)
    return rng.random((B, N, 3), dtype=np.float32)


def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    """Uniform rotation on SO(3) from a normalised Gaussian quaternion."""
    q = rng.normal(size=4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


def _sphere_surface(rng, n, radius):
    v = rng.normal(size=(n, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    return v * radius


def _box_surface(rng, n, half):
    # faces chosen with probability proportional to their area
    hx, hy, hz = half
    areas = np.array([hy * hz, hy * hz, hx * hz, hx * hz, hx * hy, hx * hy])
    face = rng.choice(6, size=n, p=areas / areas.sum())
    u = rng.uniform(-1.0, 1.0, size=(n, 2))
    p = np.empty((n, 3))
    ax = face // 2
    sign = np.where(face % 2 == 0, -1.0, 1.0)
    for a in range(3):
        others = [i for i in range(3) if i != a]
        sel = ax == a
        p[sel, a] = sign[sel] * half[a]
        p[sel, others[0]] = u[sel, 0] * half[others[0]]
        p[sel, others[1]] = u[sel, 1] * half[others[1]]
    return p


def _cylinder_surface(rng, n, radius, half_h):
    side = 2 * np.pi * radius * 2 * half_h
    cap = np.pi * radius * radius
    part = rng.choice(3, size=n, p=np.array([side, cap, cap]) / (side + 2 * cap))
    th = rng.uniform(0, 2 * np.pi, size=n)
    p = np.empty((n, 3))
    s = part == 0
    p[s, 0] = radius * np.cos(th[s])
    p[s, 1] = radius * np.sin(th[s])
    p[s, 2] = rng.uniform(-half_h, half_h, size=s.sum())
    c = ~s
    rr = radius * np.sqrt(rng.uniform(0, 1, size=c.sum()))
    p[c, 0] = rr * np.cos(th[c])
    p[c, 1] = rr * np.sin(th[c])
    p[c, 2] = np.where(part[c] == 1, -half_h, half_h)
    return p


def object_clouds(B: int, N: int, seed: int) -> np.ndarray:
    """ModelNet-like objects: 1-4 posed primitives, unit-sphere normalised."""
    rng = np.random.default_rng(seed)
    out = np.empty((B, N, 3), dtype=np.float32)
    for b in range(B):
        nprim = int(rng.integers(1, 5))
        kinds = rng.integers(0, 3, size=nprim)
        scales = rng.uniform(0.3, 1.0, size=(nprim, 3))
        areas = []
        for k, sc in zip(kinds, scales):
            if k == 0:
                areas.append(4 * np.pi * sc[0] ** 2)
            elif k == 1:
                hx, hy, hz = sc / 2
                areas.append(8 * (hx * hy + hy * hz + hx * hz))
            else:
                rad, hh = sc[0] / 2, sc[2] / 2
                areas.append(2 * np.pi * rad * 2 * hh + 2 * np.pi * rad * rad)
        areas = np.asarray(areas)
        counts = rng.multinomial(N, areas / areas.sum())
        parts = []
        for k, sc, cnt in zip(kinds, scales, counts):
            if cnt == 0:
                continue
            if k == 0:
                p = _sphere_surface(rng, cnt, sc[0])
            elif k == 1:
                p = _box_surface(rng, cnt, sc / 2)
            else:
                p = _cylinder_surface(rng, cnt, sc[0] / 2, sc[2] / 2)
            p = p @ _random_rotation(rng).T + rng.uniform(-0.7, 0.7, size=3)
            parts.append(p)
        pts = np.concatenate(parts, axis=0)
        pts -= pts.mean(axis=0)
        pts /= np.linalg.norm(pts, axis=1).max()
        pts += rng.normal(0.0, 0.005, size=pts.shape)
        pts = pts[rng.permutation(N)]
        out[b] = pts.astype(np.float32)
    return out


def _room_surfaces(rng, size_xy, height, nbox_range):
    """List of (kind, params, area) planar rectangles making up a room."""
    L = size_xy
    rects = []  # (origin, u, v): point = o + a*u + b*v, a,b in [0,1)

    def add(o, u, v):
        rects.append((np.asarray(o, float), np.asarray(u, float), np.asarray(v, float)))

    add([0, 0, 0], [L, 0, 0], [0, L, 0])                # floor
    add([0, 0, 0], [L, 0, 0], [0, 0, height])           # wall y=0
    add([0, L, 0], [L, 0, 0], [0, 0, height])           # wall y=L
    add([0, 0, 0], [0, L, 0], [0, 0, height])           # wall x=0
    add([L, 0, 0], [0, L, 0], [0, 0, height])           # wall x=L
    nbox = int(rng.integers(nbox_range[0], nbox_range[1] + 1))
    for _ in range(nbox):
        fx, fy = rng.uniform(0.2, 1.5, size=2)
        h = rng.uniform(0.2, 2.0)
        x0 = rng.uniform(0.0, L - fx)
        y0 = rng.uniform(0.0, L - fy)
        add([x0, y0, h], [fx, 0, 0], [0, fy, 0])          # top
        add([x0, y0, 0], [fx, 0, 0], [0, 0, h])           # side y0
        add([x0, y0 + fy, 0], [fx, 0, 0], [0, 0, h])      # side y1
        add([x0, y0, 0], [0, fy, 0], [0, 0, h])           # side x0
        add([x0 + fx, y0, 0], [0, fy, 0], [0, 0, h])      # side x1
    return rects


def _room_one(rng, N, size_xy, height, nbox_range, noise):
    rects = _room_surfaces(rng, size_xy, height, nbox_range)
    areas = np.array([np.linalg.norm(np.cross(u, v)) for _, u, v in rects])
    prob = areas / areas.sum()
    sensor = np.array([rng.uniform(0.5, size_xy - 0.5),
                       rng.uniform(0.5, size_xy - 0.5),
                       rng.uniform(1.0, 2.0)])
    origins = np.stack([r[0] for r in rects])
    us = np.stack([r[1] for r in rects])
    vs = np.stack([r[2] for r in rects])
    got = []
    have = 0
    while have < N:
        m = 4 * N
        ridx = rng.choice(len(rects), size=m, p=prob)
        ab = rng.random((m, 2))
        p = origins[ridx] + ab[:, :1] * us[ridx] + ab[:, 1:] * vs[ridx]
        d = np.linalg.norm(p - sensor, axis=1)
        keep = rng.random(m) < np.minimum(1.0, 1.0 / np.maximum(d, 1e-6) ** 2)
        p = p[keep]
        got.append(p)
        have += len(p)
    pts = np.concatenate(got, axis=0)[:N]
    pts = pts + rng.normal(0.0, noise, size=pts.shape)
    return pts[rng.permutation(N)]


def room_scenes(B: int, N: int, seed: int, size_xy: float = 6.0,
                height: float = 3.0, nbox_range=(10, 30), noise: float = 0.01) -> np.ndarray:
    """ScanNet-like rooms: floor, walls, boxes; density ~ min(1, (1 m / d)^2)."""
    rng = np.random.default_rng(seed)
    out = np.empty((B, N, 3), dtype=np.float32)
    for b in range(B):
        out[b] = _room_one(rng, N, size_xy, height, nbox_range, noise).astype(np.float32)
    return out


def big_room_scenes(B: int, N: int, seed: int) -> np.ndarray:
    """Full indoor scenes: 8 m x 8 m x 3 m, 20-60 boxes."""
    return room_scenes(B, N, seed, size_xy=8.0, height=3.0, nbox_range=(20, 60), noise=0.01)


def lidar_sweep(B: int, N: int, seed: int, rings: int = 64, az_steps: int = 2048,
                sweeps: int = 8, max_range: float = 80.0, nboxes: int = 200) -> np.ndarray:
    """64-ring spinning sensor 1.8 m above a ground plane with random boxes.

    Elevations are linear in [-25, +3] degrees; sweep s is offset by s/8 of an
    azimuth step. Rays are cast against the ground and axis-aligned boxes
    (each box is tested only against the rays inside its azimuth span); rays
    that hit nothing return at ``max_range``. Range noise sigma 0.02 m.
    Points are kept in scan order (sweep, ring, azimuth).
    """
    assert N == rings * az_steps * sweeps, "lidar sweep size is fixed by its scan pattern"
    rng = np.random.default_rng(seed)
    out = np.empty((B, N, 3), dtype=np.float32)
    h = 1.8
    elev = np.deg2rad(np.linspace(-25.0, 3.0, rings))
    ce, se = np.cos(elev), np.sin(elev)
    for b in range(B):
        # boxes resting on the ground, centres uniform in the disc 3 m < r < max_range,
        # rejected when their footprint comes within 1.5 m of the sensor
        boxes = []
        while len(boxes) < nboxes:
            r = max_range * np.sqrt(rng.uniform((3.0 / max_range) ** 2, 1.0))
            th = rng.uniform(0, 2 * np.pi)
            cx, cy = r * np.cos(th), r * np.sin(th)
            sx, sy, sz = rng.uniform(1.0, 8.0), rng.uniform(1.0, 3.0), rng.uniform(1.0, 3.5)
            dx = max(abs(cx) - sx / 2, 0.0)
            dy = max(abs(cy) - sy / 2, 0.0)
            if np.hypot(dx, dy) < 1.5:
                continue
            boxes.append((cx - sx / 2, cy - sy / 2, -h, cx + sx / 2, cy + sy / 2, -h + sz))
        boxes = np.asarray(boxes)
        pts = np.empty((sweeps, rings, az_steps, 3))
        for s in range(sweeps):
            az = 2 * np.pi * (np.arange(az_steps) + s / sweeps) / az_steps
            dirs = np.empty((rings, az_steps, 3))
            dirs[..., 0] = ce[:, None] * np.cos(az)[None, :]
            dirs[..., 1] = ce[:, None] * np.sin(az)[None, :]
            dirs[..., 2] = se[:, None]
            t = np.full((rings, az_steps), max_range)
            down = dirs[..., 2] < 0
            tg = np.where(down, -h / np.where(down, dirs[..., 2], -1.0), np.inf)
            t = np.minimum(t, tg)
            for k in range(nboxes):
                x0, y0, z0, x1, y1, z1 = boxes[k]
                cang = np.arctan2((y0 + y1) / 2, (x0 + x1) / 2)
                corners = np.arctan2([y0, y0, y1, y1], [x0, x1, x0, x1]) - cang
                corners = (corners + np.pi) % (2 * np.pi) - np.pi
                lo, hi = cang + corners.min(), cang + corners.max()
                i0 = int(np.floor(lo / (2 * np.pi) * az_steps - s / sweeps)) - 1
                i1 = int(np.ceil(hi / (2 * np.pi) * az_steps - s / sweeps)) + 1
                idx = np.arange(i0, i1 + 1) % az_steps
                d = dirs[:, idx, :]
                inv = 1.0 / np.where(np.abs(d) < 1e-12, 1e-12, d)
                bmin = np.array([x0, y0, z0])
                bmax = np.array([x1, y1, z1])
                t1 = bmin * inv
                t2 = bmax * inv
                tn = np.minimum(t1, t2).max(axis=-1)
                tf = np.maximum(t1, t2).min(axis=-1)
                hit = (tf >= tn) & (tn > 0)
                cur = t[:, idx]
                t[:, idx] = np.where(hit & (tn < cur), tn, cur)
            t = t + rng.normal(0.0, 0.02, size=t.shape)
            pts[s] = dirs * t[..., None]
        out[b] = pts.reshape(-1, 3).astype(np.float32)
    return out


_GENERATORS = {
    "tiny": uniform_cube,
    "object": object_clouds,
    "room": room_scenes,
    "bigroom": big_room_scenes,
    "lidar": lidar_sweep,
}


# ---------------------------------------------------------------------------
# the five workloads (grid parameters are part of the workload definition)
# ---------------------------------------------------------------------------

def _g(o, s, dims, n_v, r=1):
    return GridSpec(tuple(float(np.float32(x)) for x in o),
                    tuple(float(np.float32(x)) for x in s), tuple(dims), n_v, r)


_ROOM4 = [
    (_g((-0.2,) * 3, (0.05,) * 3, (168, 168, 68), 32), 8192),
    (_g((-0.2,) * 3, (0.1,) * 3, (84, 84, 34), 32), 2048),
    (_g((-0.2,) * 3, (0.2,) * 3, (42, 42, 17), 32), 512),
    (_g((-0.2,) * 3, (0.4,) * 3, (21, 21, 9), 32), 128),
]

WORKLOADS = {
    "tiny": Workload(
        "tiny", 1, 1024,
        (LayerSpec(_g((0, 0, 0), (0.025,) * 3, (40, 40, 40), 8), 128, 16, "rvs", "cube", 42),),
        1001, "B=1, N=1024 uniform in [0,1)^3, 40^3 grid, n_v=8, RVS M=128, cube K=16"),
    "object": Workload(
        "object", 16, 1024,
        (LayerSpec(_g((-1, -1, -1), (0.05,) * 3, (40, 40, 40), 16), 512, 32, "cas", "knn", 42),
         LayerSpec(_g((-1, -1, -1), (0.05,) * 3, (40, 40, 40), 16), 128, 32, "rvs", "cube", 43)),
        1002, "B=16 objects x 1024 pts, 40^3 grid, n_v=16; L1 CAS M=512 kNN K=32; L2 RVS M=128 cube K=32"),
    "room": Workload(
        "room", 8, 8192,
        (LayerSpec(_g((-0.2,) * 3, (0.1,) * 3, (64, 64, 34), 32), 1024, 32, "cas", "knn", 42),),
        1003, "B=8 rooms x 8192 pts, 0.1 m voxels, n_v=32, CAS M=1024 kNN K=32"),
    "bigroom/cas-knn": Workload(
        "bigroom/cas-knn", 4, 81920,
        tuple(LayerSpec(g, m, 32, "cas", "knn", 42 + i) for i, (g, m) in enumerate(_ROOM4)),
        1004, "B=4 scenes x 81920 pts, 4 layers (0.05/0.1/0.2/0.4 m; M=8192/2048/512/128), K=32, CAS+kNN"),
    "bigroom/rvs-cube": Workload(
        "bigroom/rvs-cube", 4, 81920,
        tuple(LayerSpec(g, m, 32, "rvs", "cube", 42 + i) for i, (g, m) in enumerate(_ROOM4)),
        1004, "B=4 scenes x 81920 pts, 4 layers (0.05/0.1/0.2/0.4 m; M=8192/2048/512/128), K=32, RVS+cube"),
    "lidar": Workload(
        "lidar", 1, 1048576,
        (LayerSpec(_g((-80.2, -80.2, -2.2), (0.2,) * 3, (802, 802, 33), 64, 2), 16384, 32, "rvs", "cube", 42),),
        1005, "B=1, 2^20 pts, 64-ring sweep, 0.2 m voxels, n_v=64, r=2, RVS M=16384, cube K=32"),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def small_variants() -> List[str]:
    return ["tiny", "object", "room"]

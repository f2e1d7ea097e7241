"""Seeded synthetic point clouds and embeddings for the partition workloads.

This module holds input generation only -- none of the partition method's
arithmetic -- and is the one piece both the GPU path's tests and the oracle's
tests consume.  Scenes stand in for the paper's datasets (S3DIS, KITTI-360,
DALES; Sec. 4.1), which are not available: each scene is built from planar,
box, cylinder, heightfield and blob primitives, and every point's embedding is
its primitive's constant vector drawn N(0, I_D) plus N(0, sigma^2) noise, the
structure the learned embeddings of Sec. 3.1 are trained to have
(homogeneous inside objects, contrasted across them).

Every draw uses ``numpy.random.default_rng(seed)`` (PCG64) in a fixed order,
so a scene is a pure function of its name and seed.
"""
from __future__ import annotations

import hashlib
import os
from dataclasses import dataclass, field

import numpy as np

NOISE_XYZ = 0.005  # 5 mm position noise in every scene


@dataclass
class Scene:
    name: str
    xyz: np.ndarray          # [n, 3] float32
    emb: np.ndarray          # [n, d] float32
    obj: np.ndarray          # [n] int32 primitive id (diagnostics only)
    k: int
    lambdas: list = field(default_factory=list)
    min_size: list | None = None  # s_min per level (None: off)

    @property
    def n(self) -> int:
        return self.xyz.shape[0]

    @property
    def d(self) -> int:
        return self.emb.shape[1]

    def digest(self) -> str:
        h = hashlib.sha256()
        h.update(self.xyz.tobytes())
        h.update(self.emb.tobytes())
        return h.hexdigest()[:16]


# --------------------------------------------------------------------------
# primitive samplers (area-uniform)
# --------------------------------------------------------------------------

def _rect(rng, m, origin, u, v):
    """m points uniform on the parallelogram origin + a*u + b*v, a,b in [0,1)."""
    a = rng.random(m)[:, None]
    b = rng.random(m)[:, None]
    return origin[None, :] + a * u[None, :] + b * v[None, :]


def _box_faces(lo, hi):
    """The 5 faces of an axis-aligned box resting on its bottom face
    (bottom excluded): list of (origin, u, v, area)."""
    dx, dy, dz = hi - lo
    ex, ey, ez = np.array([dx, 0, 0.]), np.array([0, dy, 0.]), \
        np.array([0, 0, dz])
    faces = [
        (np.array([lo[0], lo[1], hi[2]]), ex, ey, dx * dy),   # top
        (lo.copy(), ex, ez, dx * dz),                          # y = lo
        (np.array([lo[0], hi[1], lo[2]]), ex, ez, dx * dz),   # y = hi
        (lo.copy(), ey, ez, dy * dz),                          # x = lo
        (np.array([hi[0], lo[1], lo[2]]), ey, ez, dy * dz),   # x = hi
    ]
    return faces


def _sample_faces(rng, faces, m):
    areas = np.array([f[3] for f in faces])
    cnt = rng.multinomial(m, areas / areas.sum())
    parts = [_rect(rng, c, f[0], f[1], f[2]) for f, c in zip(faces, cnt)]
    return np.concatenate(parts, 0) if parts else np.zeros((0, 3))


def _embed(rng, obj, n_obj, d, sigma):
    centers = rng.standard_normal((n_obj, d))
    noise = rng.standard_normal((obj.shape[0], d)) * sigma
    return (centers[obj] + noise).astype(np.float32)


def _finish(rng, name, pts, obj, d, sigma, k, lambdas, shuffle=True):
    pts = pts + rng.standard_normal(pts.shape) * NOISE_XYZ
    n_obj = int(obj.max()) + 1
    emb = _embed(rng, obj, n_obj, d, sigma)
    if shuffle:
        perm = rng.permutation(pts.shape[0])
        pts, obj, emb = pts[perm], obj[perm], emb[perm]
    return Scene(name, np.ascontiguousarray(pts, dtype=np.float32),
                 np.ascontiguousarray(emb), obj.astype(np.int32), k,
                 [float(x) for x in lambdas])


# --------------------------------------------------------------------------
# indoor rooms
# --------------------------------------------------------------------------

def _room_primitives(rng, size, n_boxes):
    """Room shell (6 planes) and n_boxes boxes standing on the floor."""
    X, Y, Z = size
    prims = [
        [(np.zeros(3), np.array([X, 0, 0.]), np.array([0, Y, 0.]), X * Y)],
        [(np.array([0, 0, Z]), np.array([X, 0, 0.]), np.array([0, Y, 0.]),
          X * Y)],
        [(np.zeros(3), np.array([X, 0, 0.]), np.array([0, 0, Z]), X * Z)],
        [(np.array([0, Y, 0.]), np.array([X, 0, 0.]), np.array([0, 0, Z]),
          X * Z)],
        [(np.zeros(3), np.array([0, Y, 0.]), np.array([0, 0, Z]), Y * Z)],
        [(np.array([X, 0, 0.]), np.array([0, Y, 0.]), np.array([0, 0, Z]),
          Y * Z)],
    ]
    for _ in range(n_boxes):
        s = rng.uniform(0.3, 1.5, 3)
        s[2] = min(s[2], Z - 0.05)
        x0 = rng.uniform(0.0, X - s[0])
        y0 = rng.uniform(0.0, Y - s[1])
        lo = np.array([x0, y0, 0.0])
        prims.append(_box_faces(lo, lo + s))
    return prims


def _sample_room(rng, prims, m):
    areas = np.array([sum(f[3] for f in p) for p in prims])
    cnt = rng.multinomial(m, areas / areas.sum())
    pts, obj = [], []
    for i, (p, c) in enumerate(zip(prims, cnt)):
        pts.append(_sample_faces(rng, p, c))
        obj.append(np.full(c, i, np.int32))
    return np.concatenate(pts, 0), np.concatenate(obj, 0)


def room_small(seed: int = 0) -> Scene:
    """Indoor room, 20,000 points: 6 planes of a 5x5x3 m box plus 10 boxes;
    D = 8, embedding noise 0.05; k = 10; lambda = 0.1."""
    rng = np.random.default_rng(seed)
    prims = _room_primitives(rng, (5.0, 5.0, 3.0), 10)
    pts, obj = _sample_room(rng, prims, 20_000)
    return _finish(rng, "room-20k", pts, obj, 8, 0.05, 10, [0.1])


def room_1m(seed: int = 0) -> Scene:
    """Indoor room, 1,000,000 points after 2 cm voxel subsampling: 40
    primitives (6 planes + 34 boxes) in a 10x8x3 m volume; D = 16, embedding
    noise 0.05; k = 10; lambda ladder {0.05, 0.2, 0.8}."""
    rng = np.random.default_rng(seed)
    prims = _room_primitives(rng, (10.0, 8.0, 3.0), 34)
    m = 6_000_000
    while True:
        pts, obj = _sample_room(rng, prims, m)
        pts = pts + rng.standard_normal(pts.shape) * NOISE_XYZ
        # 2 cm grid subsampling: keep the lowest-index point of each voxel
        vox = np.floor(pts / 0.02).astype(np.int64)
        vox -= vox.min(0)
        key = (vox[:, 0] * (vox[:, 1].max() + 1) + vox[:, 1]) * \
            (vox[:, 2].max() + 1) + vox[:, 2]
        _, first = np.unique(key, return_index=True)
        if first.shape[0] >= 1_000_000:
            break
        m *= 2
    keep = np.sort(rng.choice(first, 1_000_000, replace=False))
    pts, obj = pts[keep], obj[keep]
    n_obj = int(obj.max()) + 1
    emb = _embed(rng, obj, n_obj, 16, 0.05)
    perm = rng.permutation(pts.shape[0])
    return Scene("room-1m", np.ascontiguousarray(pts[perm], np.float32),
                 np.ascontiguousarray(emb[perm]), obj[perm].astype(np.int32),
                 10, [0.05, 0.2, 0.8])


# --------------------------------------------------------------------------
# driving tile (mobile LiDAR stand-in)
# --------------------------------------------------------------------------

def _heightfield(rng, n_waves, wl_lo, wl_hi, amp):
    th = rng.uniform(0, 2 * np.pi, n_waves)
    wl = rng.uniform(wl_lo, wl_hi, n_waves)
    ph = rng.uniform(0, 2 * np.pi, n_waves)
    a = amp / n_waves

    def h(x, y):
        z = np.zeros(np.broadcast(x, y).shape)
        for j in range(n_waves):
            z += a * np.sin(2 * np.pi * (x * np.cos(th[j]) + y * np.sin(th[j]))
                            / wl[j] + ph[j])
        return z
    return h


def _density(x, y):
    """Relative point density of a sensor at the origin: 1/max(r, 2 m)^2,
    scaled to 1 inside the 2 m disk."""
    r = np.hypot(x, y)
    return (2.0 / np.maximum(r, 2.0)) ** 2


def _rect_min_range(x0, x1, y0, y1):
    dx = max(x0, 0.0, -x1)
    dy = max(y0, 0.0, -y1)
    return np.hypot(dx, dy)


def _street(rng, half):
    """The street scene of the driving tile: ground heightfield (8
    sinusoids, wavelengths 10-50 m, 1 m peak) and 200 car boxes, 300 poles
    (r = 0.15 m) and 40 facade rectangles inside [-half, half]^2, as
    (h, objects) with objects[i] = (kind, params) for object id i + 1 (the
    ground is object 0)."""
    h = _heightfield(rng, 8, 10.0, 50.0, 1.0)
    objs = []
    for _ in range(200):  # cars: ~4.5 x 1.8 x 1.5 m, +-10 %, axis-aligned
        s = np.array([4.5, 1.8, 1.5]) * rng.uniform(0.9, 1.1, 3)
        if rng.random() < 0.5:
            s[0], s[1] = s[1], s[0]
        c = rng.uniform(-half + 3, half - 3, 2)
        lo = np.array([c[0] - s[0] / 2, c[1] - s[1] / 2, float(h(c[0], c[1]))])
        objs.append(("box", lo, lo + s))
    for _ in range(300):  # poles
        c = rng.uniform(-half + 1, half - 1, 2)
        ht = rng.uniform(3.0, 8.0)
        objs.append(("pole", np.array([c[0], c[1], float(h(c[0], c[1]))]), ht))
    for _ in range(40):  # facades: vertical rectangles
        wdt = rng.uniform(10.0, 40.0)
        ht = rng.uniform(5.0, 15.0)
        c = rng.uniform(-half + 5, half - 5, 2)
        along_x = rng.random() < 0.5
        z0 = float(h(c[0], c[1]))
        if along_x:
            o = np.array([c[0] - wdt / 2, c[1], z0])
            u = np.array([wdt, 0, 0.])
        else:
            o = np.array([c[0], c[1] - wdt / 2, z0])
            u = np.array([0, wdt, 0.])
        objs.append(("facade", o, u, np.array([0, 0, ht])))
    return h, objs


def driving_tile(seed: int = 0, n_points: int = 3_000_000) -> Scene:
    """Driving tile, 3,000,000 points: ground heightfield (8 sinusoids,
    wavelengths 10-50 m, 1 m peak) over 100x100 m, 200 car boxes, 300 poles
    (r = 0.15 m), 40 facade planes; density 1/max(r, 2 m)^2 around a sensor at
    the origin; D = 16, embedding noise 0.05; k = 10; ladder {0.05, 0.2,
    0.8}."""
    rng = np.random.default_rng(seed)
    half = 50.0
    h, objs = _street(rng, half)

    def obj_surface(ob, m):
        if ob[0] == "box":
            return _sample_faces(rng, _box_faces(ob[1], ob[2]), m)
        if ob[0] == "pole":
            base, ht = ob[1], ob[2]
            t = rng.uniform(0, 2 * np.pi, m)
            z = rng.uniform(0, ht, m)
            return np.stack([base[0] + 0.15 * np.cos(t),
                             base[1] + 0.15 * np.sin(t), base[2] + z], 1)
        return _rect(rng, m, ob[1], ob[2], ob[3])

    def obj_area_pmax(ob):
        if ob[0] == "box":
            lo, hi = ob[1], ob[2]
            area = sum(f[3] for f in _box_faces(lo, hi))
            r = _rect_min_range(lo[0], hi[0], lo[1], hi[1])
        elif ob[0] == "pole":
            area = 2 * np.pi * 0.15 * ob[2]
            r = max(np.hypot(ob[1][0], ob[1][1]) - 0.15, 0.0)
        else:
            p0, p1 = ob[1][:2], ob[1][:2] + ob[2][:2]
            area = np.linalg.norm(ob[2]) * ob[3][2]
            r = _rect_min_range(min(p0[0], p1[0]), max(p0[0], p1[0]),
                                min(p0[1], p1[1]), max(p0[1], p1[1]))
        return area, (2.0 / max(r, 2.0)) ** 2

    # density integrals: ground over the tile by the radial law; objects by
    # a pilot Monte-Carlo pass
    R = half * np.sqrt(2.0)
    disk_int = 4 * np.pi + 8 * np.pi * np.log(R / 2.0)  # density over the disk
    pilot = rng.uniform(-half, half, (200_000, 2))
    ground_int = (2 * half) ** 2 * _density(pilot[:, 0], pilot[:, 1]).mean()
    obj_int = []
    for ob in objs:
        q = obj_surface(ob, 512)
        area, _ = obj_area_pmax(ob)
        obj_int.append(area * _density(q[:, 0], q[:, 1]).mean())
    K = 1.04 * n_points / (ground_int + sum(obj_int))  # points per unit

    # ground: radial inverse-CDF sampling, rejected outside the square
    m_g = int(round(K * disk_int))
    u = rng.random(m_g) * (0.5 + np.log(R / 2.0))
    r = np.where(u < 0.5, np.sqrt(8.0 * u), 2.0 * np.exp(u - 0.5))
    t = rng.uniform(0, 2 * np.pi, m_g)
    gx, gy = r * np.cos(t), r * np.sin(t)
    inside = (np.abs(gx) < half) & (np.abs(gy) < half)
    gx, gy = gx[inside], gy[inside]
    pts = [np.stack([gx, gy, h(gx, gy)], 1)]
    obj = [np.zeros(gx.shape[0], np.int32)]
    for i, ob in enumerate(objs):
        area, pmax = obj_area_pmax(ob)
        m = int(np.ceil(K * area * pmax))
        q = obj_surface(ob, m)
        acc = rng.random(m) < _density(q[:, 0], q[:, 1]) / pmax
        pts.append(q[acc])
        obj.append(np.full(int(acc.sum()), i + 1, np.int32))
    pts = np.concatenate(pts, 0)
    obj = np.concatenate(obj, 0)
    if pts.shape[0] < n_points:
        raise RuntimeError("driving tile generator undershot: %d" % pts.shape[0])
    keep = np.sort(rng.choice(pts.shape[0], n_points, replace=False))
    return _finish(rng, "driving-3m", pts[keep], obj[keep], 16, 0.05, 10,
                   [0.05, 0.2, 0.8])


# --------------------------------------------------------------------------
# aerial tile (airborne LiDAR stand-in)
# --------------------------------------------------------------------------

def aerial_tile(seed: int = 0, n_points: int = 10_000_000) -> Scene:
    """Aerial tile, 10,000,000 points: 500x500 m terrain (5 m amplitude,
    wavelengths 50-200 m), 400 non-overlapping buildings (footprint 10-40 m,
    height 5-30 m), 2000 Gaussian vegetation blobs; 90 % of points top-down
    uniform (roof or terrain), 10 % in blobs (about 40 pts/m^2); D = 16,
    embedding noise 0.1; k = 10; ladder {0.05, 0.2, 0.8, 3.2}."""
    rng = np.random.default_rng(seed)
    S = 500.0
    h = _heightfield(rng, 8, 50.0, 200.0, 5.0)
    grid = -np.ones((500, 500), np.int32)  # 1 m raster of building ids
    bld = []
    tries = 0
    while len(bld) < 400 and tries < 100_000:
        tries += 1
        w, l = rng.uniform(10, 40, 2)
        x0, y0 = rng.uniform(0, S - w), rng.uniform(0, S - l)
        i0, i1 = int(np.floor(x0)), int(np.ceil(x0 + w))
        j0, j1 = int(np.floor(y0)), int(np.ceil(y0 + l))
        if (grid[i0:i1, j0:j1] >= 0).any():
            continue
        ht = rng.uniform(5, 30)
        roof = float(h(x0 + w / 2, y0 + l / 2)) + ht
        grid[i0:i1, j0:j1] = len(bld)
        bld.append((x0, y0, w, l, roof))
    roof_z = np.array([b[4] for b in bld])
    n_top = int(round(0.9 * n_points))
    x = rng.uniform(0, S, n_top)
    y = rng.uniform(0, S, n_top)
    b = grid[np.minimum(x.astype(np.int64), 499), np.minimum(y.astype(np.int64), 499)]
    # exact footprint test inside the raster cells that carry a building id
    bx0 = np.array([q[0] for q in bld]); by0 = np.array([q[1] for q in bld])
    bw = np.array([q[2] for q in bld]); bl = np.array([q[3] for q in bld])
    on = b >= 0
    bb = np.where(on, b, 0)
    on &= (x >= bx0[bb]) & (x < bx0[bb] + bw[bb]) & (y >= by0[bb]) & \
        (y < by0[bb] + bl[bb])
    z = np.where(on, roof_z[bb], h(x, y))
    obj_top = np.where(on, 1 + bb, 0).astype(np.int32)
    n_blob = n_points - n_top
    bc = np.stack([rng.uniform(0, S, 2000), rng.uniform(0, S, 2000)], 1)
    bz = h(bc[:, 0], bc[:, 1]) + rng.uniform(3, 10, 2000)
    bs = rng.uniform(1, 3, 2000)
    which = rng.integers(0, 2000, n_blob)
    off = rng.standard_normal((n_blob, 3)) * bs[which][:, None]
    blob = np.stack([bc[which, 0], bc[which, 1], bz[which]], 1) + off
    pts = np.concatenate([np.stack([x, y, z], 1), blob], 0)
    obj = np.concatenate([obj_top, (1 + len(bld) + which).astype(np.int32)])
    return _finish(rng, "aerial-10m", pts, obj, 16, 0.1, 10,
                   [0.05, 0.2, 0.8, 3.2])


# --------------------------------------------------------------------------
# the paper's own partition settings on the same geometry (Sec. 4.1:
# embeddings of dimension 32, 8 nearest neighbours, one lambda = 0.02 and
# minimal superpoint sizes [5, 30, 90] for the indoor and mobile-mapping
# data, [5, 15, 70] for the aerial data)
# --------------------------------------------------------------------------

def _paper_variant(base, name, sigma, min_size, seed):
    """The base scene's points and primitives with D = 32 embeddings drawn
    from their own generator stream (the base scene's draws are untouched)."""
    sc = base(seed)
    rng = np.random.default_rng([seed, 32])
    n_obj = int(sc.obj.max()) + 1
    emb = np.ascontiguousarray(_embed(rng, sc.obj, n_obj, 32, sigma))
    return Scene(name, sc.xyz, emb, sc.obj, 8, [0.02, 0.02, 0.02],
                 list(min_size))


def room_small_paper(seed: int = 0) -> Scene:
    return _paper_variant(room_small, "room-20k-paper", 0.05, [5, 30, 90],
                          seed)


def room_1m_paper(seed: int = 0) -> Scene:
    return _paper_variant(room_1m, "room-1m-paper", 0.05, [5, 30, 90], seed)


def driving_tile_paper(seed: int = 0) -> Scene:
    return _paper_variant(driving_tile, "driving-3m-paper", 0.05, [5, 30, 90],
                          seed)


def aerial_tile_paper(seed: int = 0) -> Scene:
    return _paper_variant(aerial_tile, "aerial-10m-paper", 0.1, [5, 15, 70],
                          seed)


# --------------------------------------------------------------------------
# registry and cache
# --------------------------------------------------------------------------

SCENES = {
    "room-20k": room_small,
    "room-1m": room_1m,
    "driving-3m": driving_tile,
    "aerial-10m": aerial_tile,
    "room-20k-paper": room_small_paper,
    "room-1m-paper": room_1m_paper,
    "driving-3m-paper": driving_tile_paper,
    "aerial-10m-paper": aerial_tile_paper,
}


def _cache_dir():
    return os.environ.get("EZSP_SCENE_CACHE", "/tmp/ezsp_scenes")


def load(name: str, seed: int = 0, cache: bool = True) -> Scene:
    """Generate (or read back from the on-disk cache) a named scene."""
    path = os.path.join(_cache_dir(), f"{name}-s{seed}.npz")
    if cache and os.path.exists(path):
        z = np.load(path, allow_pickle=False)
        ms = (z["min_size"] if "min_size" in z.files
              else np.zeros(0, np.int64))
        return Scene(name, z["xyz"], z["emb"], z["obj"], int(z["k"]),
                     [float(x) for x in z["lambdas"]],
                     [int(x) for x in ms] if ms.size else None)
    sc = SCENES[name](seed)
    if cache:
        os.makedirs(_cache_dir(), exist_ok=True)
        tmp = path + ".tmp%d.npz" % os.getpid()
        np.savez(tmp, xyz=sc.xyz, emb=sc.emb, obj=sc.obj, k=sc.k,
                 lambdas=np.array(sc.lambdas),
                 min_size=np.array(sc.min_size or [], np.int64))
        os.replace(tmp, path)
    return sc


def random_cloud(n: int, d: int, seed: int = 0, n_obj: int = 8,
                 sigma: float = 0.05, extent: float = 1.0) -> Scene:
    """Small unstructured cloud: n_obj Gaussian clusters with constant
    embeddings plus noise (test inputs of any size)."""
    rng = np.random.default_rng(seed)
    c = rng.uniform(0, extent, (n_obj, 3))
    obj = rng.integers(0, n_obj, n).astype(np.int32)
    xyz = c[obj] + rng.standard_normal((n, 3)) * (0.1 * extent)
    emb = _embed(rng, obj, n_obj, d, sigma)
    return Scene(f"random-{n}", xyz.astype(np.float32), emb, obj, 10, [0.1])


# --------------------------------------------------------------------------
# LiDAR sweep (the streaming workload): one revolution of a 64-beam rotating
# sensor ray-cast against the driving tile's street scene, stored ring-major
# (every azimuth of ring 0, then ring 1, ...), the order in which a scanning
# sensor's points arrive once sorted by laser.  Per-point features
# [x/50, y/50, z/5, intensity, range/120, ring/63] in the sensor frame go
# through a random-weight MLP (PyTorch-Linear-style U(+-1/sqrt(fan_in))
# weights from default_rng(seed)); inputs and weights are handed over as
# bfloat16 bit patterns (round to nearest even).
# --------------------------------------------------------------------------

SWEEP_RINGS = 64
SWEEP_AZIMUTHS = 20_000
SWEEP_ELEV_DEG = (-24.8, 2.0)   # lowest and highest beam
SWEEP_MAX_RANGE = 120.0         # metres; farther returns are dropped
SWEEP_SENSOR_HEIGHT = 1.8       # above the ground under the sensor
SWEEP_STEP_X = 5.0              # sweep i has its sensor at x = 5 i
MLP_DIMS = (6, 32, 16)


def to_bf16_bits(a) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite)."""
    u = np.ascontiguousarray(a, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def mlp_weights(seed: int = 0, dims=MLP_DIMS):
    """(w1, b1, w2, b2, w3, b3): weights d_in x d_out as bfloat16 bits,
    biases fp32."""
    d_in, d_hid, d_out = dims
    rng = np.random.default_rng(seed)
    out = []
    for fi, fo in ((d_in, d_hid), (d_hid, d_hid), (d_hid, d_out)):
        bound = 1.0 / np.sqrt(fi)
        w = rng.uniform(-bound, bound, (fi, fo)).astype(np.float32)
        b = rng.uniform(-bound, bound, fo).astype(np.float32)
        out += [to_bf16_bits(w), b]
    return tuple(out)


def _ground_hits(h, o, dirs, tmax):
    """First intersection parameter of every ray o + t*dirs (unit
    directions, [m, 3]) with the heightfield z = h(x, y), |h| <= 1, or inf.
    The crossing lies where the ray is inside the band |z| <= 1: that part
    is marched in steps of 0.25 m of path (the heightfield's wavelengths are
    10 m and more) and the first sign change refined by 30 bisections."""
    m = dirs.shape[0]
    dz = dirs[:, 2]
    t = np.full(m, np.inf)
    with np.errstate(divide="ignore", invalid="ignore"):
        ta = np.where(dz < 0, (o[2] - 1.0) / -dz,
                      np.where(dz > 0, 0.0, 0.0))
        tb = np.where(dz < 0, (o[2] + 1.0) / -dz,
                      np.where(dz > 0, (1.0 - o[2]) / dz, np.inf))
    ta = np.maximum(ta, 0.0)
    tb = np.minimum(tb, tmax)
    live = np.nonzero(tb > ta)[0]
    step = 0.25

    def f(idx, tt):
        p = o[None, :] + tt[:, None] * dirs[idx]
        return p[:, 2] - h(p[:, 0], p[:, 1])
    lo = ta[live].copy()
    flo = f(live, lo)
    todo = flo > 0  # above the ground at the band entry
    hit_lo = np.full(live.shape[0], np.nan)
    hit_hi = np.full(live.shape[0], np.nan)
    cur = lo.copy()
    while todo.any():
        idx = np.nonzero(todo)[0]
        nxt = np.minimum(cur[idx] + step, tb[live[idx]])
        fn = f(live[idx], nxt)
        cross = fn <= 0
        hit_lo[idx[cross]] = cur[idx[cross]]
        hit_hi[idx[cross]] = nxt[cross]
        done = cross | (nxt >= tb[live[idx]])
        cur[idx] = nxt
        todo[idx[done]] = False
    ok = np.nonzero(~np.isnan(hit_lo))[0]
    a, b = hit_lo[ok], hit_hi[ok]
    for _ in range(30):
        mid = 0.5 * (a + b)
        above = f(live[ok], mid) > 0
        a = np.where(above, mid, a)
        b = np.where(above, b, mid)
    t[live[ok]] = b
    return t


def _box_hits(lo, hi, o, dirs):
    """Slab test: entry parameter of each ray into the box, or inf."""
    with np.errstate(divide="ignore", invalid="ignore"):
        inv = 1.0 / dirs
        t1 = (lo[None, :] - o[None, :]) * inv
        t2 = (hi[None, :] - o[None, :]) * inv
    t1 = np.where(np.isnan(t1), -np.inf, t1)
    t2 = np.where(np.isnan(t2), np.inf, t2)
    tn = np.minimum(t1, t2).max(1)
    tf = np.maximum(t1, t2).min(1)
    return np.where((tn <= tf) & (tn > 0), tn, np.inf)


def _pole_hits(base, ht, radius, o, dirs):
    """Entry parameter into a vertical cylinder (side only), or inf."""
    dx, dy = dirs[:, 0], dirs[:, 1]
    ox, oy = o[0] - base[0], o[1] - base[1]
    a = dx * dx + dy * dy
    b = 2 * (ox * dx + oy * dy)
    c = ox * ox + oy * oy - radius * radius
    disc = b * b - 4 * a * c
    with np.errstate(invalid="ignore", divide="ignore"):
        t = (-b - np.sqrt(disc)) / (2 * a)
    z = o[2] + t * dirs[:, 2]
    ok = (disc >= 0) & (t > 0) & (z >= base[2]) & (z <= base[2] + ht)
    return np.where(ok, t, np.inf)


def _facade_hits(orig, u, v, o, dirs):
    """Intersection with the vertical rectangle orig + a*u + b*v, a, b in
    [0, 1] (u horizontal along x or y, v vertical), or inf."""
    ax = 0 if abs(u[0]) > 0 else 1      # the axis the facade runs along
    nx = 1 - ax                          # its normal axis
    with np.errstate(divide="ignore", invalid="ignore"):
        t = (orig[nx] - o[nx]) / dirs[:, nx]
    p_a = o[ax] + t * dirs[:, ax]
    p_z = o[2] + t * dirs[:, 2]
    a = (p_a - orig[ax]) / u[ax]
    ok = (t > 0) & (a >= 0) & (a <= 1) & (p_z >= orig[2]) & \
        (p_z <= orig[2] + v[2])
    return np.where(ok, t, np.inf)


def _azimuth_span(xs, ys, o):
    """Azimuth interval (radians, start and width) seen from o that covers
    the points (xs, ys), or None when o lies inside their hull's box."""
    ang = np.arctan2(np.asarray(ys) - o[1], np.asarray(xs) - o[0])
    if (min(xs) <= o[0] <= max(xs)) and (min(ys) <= o[1] <= max(ys)):
        return None
    srt = np.sort(np.mod(ang, 2 * np.pi))
    gaps = np.diff(np.concatenate([srt, srt[:1] + 2 * np.pi]))
    j = int(np.argmax(gaps))  # the span is the complement of the widest gap
    start = srt[(j + 1) % srt.shape[0]]
    return start, 2 * np.pi - gaps[j]


SWEEP_ROAD = 8.0     # half width of the road the sensor drives along
SWEEP_CLEAR = 2.0    # clearance of objects around the sensor's path


def _blocks_road(ob, xs, ys):
    """True for a street object the sensor's road removes: a facade whose
    footprint reaches into the road |y| < 8 m, or any object within 2 m of
    the sensor path y = 0, x in [-2, 5 * 3] (the street scene places its
    objects with no regard to a road)."""
    x0, x1, y0, y1 = min(xs), max(xs), min(ys), max(ys)
    if ob[0] == "facade" and y1 > -SWEEP_ROAD and y0 < SWEEP_ROAD:
        return True
    return (x1 > -SWEEP_CLEAR and x0 < 3 * SWEEP_STEP_X + SWEEP_CLEAR and
            y1 > -SWEEP_CLEAR and y0 < SWEEP_CLEAR)


def lidar_sweep(seed: int = 0, index: int = 0):
    """Ray-cast sweep `index` of the street scene of seed `seed`.

    64 beams at elevations linspace(-24.8, +2) degrees times 20,000
    azimuths, from a sensor at (5 * index, 0) and 1.8 m above the ground
    there, driving along a road on the x axis that the street's facades
    leave free.  Each ray keeps its first hit among the ground, the cars,
    poles and facades within 120 m; rays without one are dropped.  Returns
    (xyz [n, 3] fp32 in the world frame, obj [n] int32, ring [n] int32,
    rng_m [n] fp64 range, sensor [3]); points in ring-major order, each
    with 5 mm of Gaussian position noise."""
    rng = np.random.default_rng(seed)
    h, objs = _street(rng, 50.0)
    sx = SWEEP_STEP_X * index
    o = np.array([sx, 0.0, float(h(sx, 0.0)) + SWEEP_SENSOR_HEIGHT])
    elev = np.radians(np.linspace(*SWEEP_ELEV_DEG, SWEEP_RINGS))
    azim = 2 * np.pi * np.arange(SWEEP_AZIMUTHS) / SWEEP_AZIMUTHS
    ce, se = np.cos(elev), np.sin(elev)
    dirs = np.stack([ce[:, None] * np.cos(azim)[None, :],
                     ce[:, None] * np.sin(azim)[None, :],
                     np.broadcast_to(se[:, None], (SWEEP_RINGS,
                                                   SWEEP_AZIMUTHS))],
                    -1).reshape(-1, 3)   # ring-major
    t = _ground_hits(h, o, dirs, SWEEP_MAX_RANGE)
    obj = np.zeros(t.shape[0], np.int32)
    ray_az = np.tile(np.arange(SWEEP_AZIMUTHS), SWEEP_RINGS)
    for i, ob in enumerate(objs):
        if ob[0] == "box":
            lo, hi = ob[1], ob[2]
            xs, ys = [lo[0], hi[0], lo[0], hi[0]], [lo[1], lo[1], hi[1], hi[1]]
        elif ob[0] == "pole":
            b = ob[1]
            xs = [b[0] - 0.15, b[0] + 0.15, b[0] - 0.15, b[0] + 0.15]
            ys = [b[1] - 0.15, b[1] - 0.15, b[1] + 0.15, b[1] + 0.15]
        else:
            p0, p1 = ob[1], ob[1] + ob[2]
            xs, ys = [p0[0], p1[0]], [p0[1], p1[1]]
        if _blocks_road(ob, xs, ys):
            continue
        span = _azimuth_span(xs, ys, o)
        if span is None:
            continue  # the sensor stands inside: no surface seen
        else:
            start, width = span
            a0 = int(np.floor(start / (2 * np.pi) * SWEEP_AZIMUTHS)) - 1
            a1 = int(np.ceil((start + width) / (2 * np.pi) *
                             SWEEP_AZIMUTHS)) + 1
            cols = np.mod(np.arange(a0, a1 + 1), SWEEP_AZIMUTHS)
            mask = np.zeros(SWEEP_AZIMUTHS, bool)
            mask[cols] = True
            rays = np.nonzero(mask[ray_az])[0]
        d = dirs[rays]
        if ob[0] == "box":
            ti = _box_hits(ob[1], ob[2], o, d)
        elif ob[0] == "pole":
            ti = _pole_hits(ob[1], ob[2], 0.15, o, d)
        else:
            ti = _facade_hits(ob[1], ob[2], ob[3], o, d)
        closer = ti < t[rays]
        t[rays[closer]] = ti[closer]
        obj[rays[closer]] = i + 1
    hit = np.nonzero(t <= SWEEP_MAX_RANGE)[0]   # ring-major order kept
    p = o[None, :] + t[hit, None] * dirs[hit]
    p = p + rng.standard_normal(p.shape) * NOISE_XYZ
    ring = (hit // SWEEP_AZIMUTHS).astype(np.int32)
    return (np.ascontiguousarray(p, np.float32), obj[hit], ring, t[hit], o)


def sweep_features(xyz, obj, ring, sensor, seed: int = 0):
    """The six per-point features of a sweep in the sensor frame, as
    bfloat16 bits [n, 6]: [x/50, y/50, z/5, intensity, range/120, ring/63],
    intensity = U(0, 1) per object plus N(0, 0.02^2), clipped to [0, 1]."""
    rng = np.random.default_rng([seed, 6])
    rel = np.asarray(xyz, np.float64) - np.asarray(sensor)[None, :]
    rng_m = np.sqrt((rel ** 2).sum(1))
    n_obj = int(np.max(obj)) + 1
    inten = rng.uniform(0, 1, n_obj)[obj] + rng.normal(0, 0.02, xyz.shape[0])
    feat = np.stack([rel[:, 0] / 50, rel[:, 1] / 50, rel[:, 2] / 5,
                     np.clip(inten, 0, 1), rng_m / SWEEP_MAX_RANGE,
                     np.asarray(ring, np.float64) / (SWEEP_RINGS - 1)], 1)
    return to_bf16_bits(feat.astype(np.float32))


def sweep(seed: int = 0, index: int = 0, cache: bool = True):
    """(xyz [n, 3] fp32, features [n, 6] bfloat16 bits, obj) of ray-cast
    sweep `index`; cached on disk like the scenes."""
    path = os.path.join(_cache_dir(), f"sweep{index}-s{seed}.npz")
    if cache and os.path.exists(path):
        z = np.load(path, allow_pickle=False)
        return z["xyz"], z["feat"], z["obj"]
    xyz, obj, ring, _, sensor = lidar_sweep(seed, index)
    feat = sweep_features(xyz, obj, ring, sensor, seed)
    if cache:
        os.makedirs(_cache_dir(), exist_ok=True)
        tmp = path + ".tmp%d.npz" % os.getpid()
        np.savez(tmp, xyz=xyz, feat=feat, obj=obj)
        os.replace(tmp, path)
    return xyz, feat, obj

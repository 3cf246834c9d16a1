"""Seeded synthetic point clouds shaped like the paper's workloads.

The paper evaluates on ShapeNet part objects (about 2.6k surface points per
object), ScanNet rooms (9k-537k points, 145k on average, whole rooms) and
SemanticKITTI LiDAR scans (82k-129k points, whole scans); see its
Experiments section.  None of those datasets is used here: these generators
draw clouds with the same sizes, extents and surface structure from a seeded
counter-based RNG, so the same seed always gives the same bytes.

Everything here is input preparation (positions, per-point features, layer
weights).  Nothing of the lattice method is computed in this module.
"""
from __future__ import annotations

import numpy as np

from .rng import Stream


# --------------------------------------------------------------------------
# surface primitives
# --------------------------------------------------------------------------
def _sample_sphere(st: Stream, k: int, centre, radius) -> np.ndarray:
    v = st.normal(3 * k).reshape(k, 3)
    nrm = np.linalg.norm(v, axis=1, keepdims=True)
    nrm[nrm == 0] = 1.0
    return centre + radius * v / nrm


def _box_faces(centre, half, with_bottom=True):
    """Axis-aligned box faces as (origin, edge_u, edge_v) parallelograms."""
    cx, cy, cz = centre
    hx, hy, hz = half
    x0, x1, y0, y1, z0, z1 = cx - hx, cx + hx, cy - hy, cy + hy, cz - hz, cz + hz
    faces = [
        ((x0, y0, z1), (2 * hx, 0, 0), (0, 2 * hy, 0)),   # top
        ((x0, y0, z0), (2 * hx, 0, 0), (0, 0, 2 * hz)),   # -y side
        ((x0, y1, z0), (2 * hx, 0, 0), (0, 0, 2 * hz)),   # +y side
        ((x0, y0, z0), (0, 2 * hy, 0), (0, 0, 2 * hz)),   # -x side
        ((x1, y0, z0), (0, 2 * hy, 0), (0, 0, 2 * hz)),   # +x side
    ]
    if with_bottom:
        faces.append(((x0, y0, z0), (2 * hx, 0, 0), (0, 2 * hy, 0)))
    return [tuple(np.asarray(a, dtype=np.float64) for a in f) for f in faces]


def _face_area(face) -> float:
    _, u, v = face
    return float(np.linalg.norm(np.cross(u, v)))


def _sample_faces(st: Stream, k: int, faces) -> np.ndarray:
    """k points uniform over a set of parallelogram faces (area weighted)."""
    areas = np.array([_face_area(f) for f in faces])
    cdf = np.cumsum(areas) / areas.sum()
    which = np.searchsorted(cdf, st.uniform(k), side="right")
    which = np.minimum(which, len(faces) - 1)
    a = st.uniform(k)
    b = st.uniform(k)
    out = np.empty((k, 3))
    for i, (o, u, v) in enumerate(faces):
        sel = which == i
        out[sel] = o + a[sel, None] * u + b[sel, None] * v
    return out


def _allocate(st: Stream, m: int, areas) -> np.ndarray:
    """Split m points over surfaces in proportion to area (multinomial)."""
    areas = np.asarray(areas, dtype=np.float64)
    cdf = np.cumsum(areas) / areas.sum()
    which = np.minimum(np.searchsorted(cdf, st.uniform(m), side="right"), len(areas) - 1)
    return np.bincount(which, minlength=len(areas))


# --------------------------------------------------------------------------
# clouds
# --------------------------------------------------------------------------
def uniform_cube(seed: int, m: int) -> np.ndarray:
    """m points uniform in [0,1]^3 (float32)."""
    st = Stream(seed, "cube")
    return st.uniform(3 * m).reshape(m, 3).astype(np.float32)


def object_surfaces(seed: int, m: int = 2048) -> np.ndarray:
    """A ShapeNet-sized object: m points on the surfaces of 1-4 random spheres
    or boxes, centred and scaled so that the farthest point has norm 1."""
    st = Stream(seed, "object")
    nshape = int(st.integers(1, 1, 5)[0])
    shapes = []
    for _ in range(nshape):
        centre = st.uniform_range(3, -0.5, 0.5)
        if st.uniform(1)[0] < 0.5:
            r = float(st.uniform_range(1, 0.1, 0.5)[0])
            shapes.append(("sphere", centre, r, 4.0 * np.pi * r * r))
        else:
            half = st.uniform_range(3, 0.05, 0.4)
            faces = _box_faces(centre, half, with_bottom=True)
            shapes.append(("box", centre, faces, sum(_face_area(f) for f in faces)))
    counts = _allocate(st, m, [s[3] for s in shapes])
    parts = []
    for s, k in zip(shapes, counts):
        if k == 0:
            continue
        if s[0] == "sphere":
            parts.append(_sample_sphere(st, int(k), s[1], s[2]))
        else:
            parts.append(_sample_faces(st, int(k), s[2]))
    p = np.concatenate(parts, axis=0)
    p = p - p.mean(axis=0)
    p = p / np.linalg.norm(p, axis=1).max()
    return p.astype(np.float32)


def room(seed: int, m: int, size=(8.0, 8.0, 3.0), nboxes: int = 20,
         noise: float = 0.01) -> np.ndarray:
    """An indoor room: floor, four walls and `nboxes` boxes standing on the
    floor, sampled area-weighted, plus isotropic Gaussian noise (metres).

    Points come out in the order a volumetric reconstruction emits its mesh
    vertices: block by block (0.5 m blocks in Morton order), in random order
    inside a block."""
    st = Stream(seed, "room")
    sx, sy, sz = size
    surfaces = [
        [((0, 0, 0), (sx, 0, 0), (0, sy, 0))],            # floor
        [((0, 0, 0), (sx, 0, 0), (0, 0, sz))],            # wall y=0
        [((0, sy, 0), (sx, 0, 0), (0, 0, sz))],           # wall y=sy
        [((0, 0, 0), (0, sy, 0), (0, 0, sz))],            # wall x=0
        [((sx, 0, 0), (0, sy, 0), (0, 0, sz))],           # wall x=sx
    ]
    surfaces = [[tuple(np.asarray(a, dtype=np.float64) for a in f) for f in s] for s in surfaces]
    for _ in range(nboxes):
        dims = st.uniform_range(3, 0.3, 1.5)
        half = dims / 2.0
        cxy = st.uniform_range(2, 0.0, 1.0) * (np.array([sx, sy]) - dims[:2]) + half[:2]
        centre = np.array([cxy[0], cxy[1], half[2]])
        surfaces.append(_box_faces(centre, half, with_bottom=False))
    areas = [sum(_face_area(f) for f in s) for s in surfaces]
    counts = _allocate(st, m, areas)
    parts = [_sample_faces(st, int(k), s) for s, k in zip(surfaces, counts) if k > 0]
    p = np.concatenate(parts, axis=0)
    p = p + noise * st.normal(3 * m).reshape(m, 3)
    p = p[st.permutation(m)]
    p = p[np.argsort(_morton_blocks(p, 0.5), kind="stable")]
    return p.astype(np.float32)


def _morton_blocks(p: np.ndarray, block: float) -> np.ndarray:
    """Morton (Z-order) code of the block each point falls in."""
    q = np.floor((p - p.min(axis=0)) / block).astype(np.uint64)
    code = np.zeros(p.shape[0], dtype=np.uint64)
    for bit in range(16):
        for axis in range(3):
            code |= ((q[:, axis] >> np.uint64(bit)) & np.uint64(1)) << np.uint64(3 * bit + axis)
    return code


def _ray_box(orig, dirs, lo, hi):
    """Entry distance of rays into an axis-aligned box (inf when missed)."""
    with np.errstate(divide="ignore", invalid="ignore"):
        inv = 1.0 / dirs
        t1 = (lo - orig) * inv
        t2 = (hi - orig) * inv
    tmin = np.nanmax(np.minimum(t1, t2), axis=1)
    tmax = np.nanmin(np.maximum(t1, t2), axis=1)
    hit = (tmax >= np.maximum(tmin, 0.0))
    t = np.where(tmin > 0.0, tmin, tmax)
    return np.where(hit & (t > 0.0), t, np.inf)


def lidar_scan(seed: int, m: int = 120_000, rings: int = 64, azimuths: int = 2048,
               nboxes: int = 50, max_range: float = 50.0,
               sensor_height: float = 1.73, noise: float = 0.02) -> np.ndarray:
    """A SemanticKITTI-sized spinning-LiDAR scan.

    A 64-ring sensor at height 1.73 m (elevations evenly spaced in
    [-24, -2.5] degrees, 2048 azimuth steps) casts rays at a ground plane
    z = 0 and `nboxes` random boxes; first hits within `max_range` are kept
    in firing order (azimuth-major), a seeded subset of exactly m of them is
    taken (order preserved) and 2 cm Gaussian noise is added."""
    st = Stream(seed, "lidar")
    orig = np.array([0.0, 0.0, sensor_height])
    el = np.deg2rad(np.linspace(-24.0, -2.5, rings))
    az = 2.0 * np.pi * np.arange(azimuths) / azimuths
    A, E = np.meshgrid(az, el, indexing="ij")           # azimuth-major firing order
    dirs = np.stack([np.cos(E) * np.cos(A), np.cos(E) * np.sin(A), np.sin(E)], axis=-1).reshape(-1, 3)
    t = np.where(dirs[:, 2] < 0, -sensor_height / np.where(dirs[:, 2] < 0, dirs[:, 2], -1.0), np.inf)
    for _ in range(nboxes):
        rng_c = float(st.uniform_range(1, 5.0, 45.0)[0])
        ang = float(st.uniform_range(1, 0.0, 2.0 * np.pi)[0])
        half = st.uniform_range(2, 0.5, 2.5)
        height = float(st.uniform_range(1, 1.0, 3.0)[0])
        c = np.array([rng_c * np.cos(ang), rng_c * np.sin(ang)])
        lo = np.array([c[0] - half[0], c[1] - half[1], 0.0])
        hi = np.array([c[0] + half[0], c[1] + half[1], height])
        t = np.minimum(t, _ray_box(orig, dirs, lo, hi))
    keep = np.isfinite(t) & (t <= max_range)
    pts = orig + dirs[keep] * t[keep, None]
    if pts.shape[0] < m:
        raise ValueError(f"scan produced {pts.shape[0]} hits < {m}")
    sel = np.sort(st.permutation(pts.shape[0])[:m])
    pts = pts[sel] + noise * st.normal(3 * m).reshape(m, 3)
    return pts.astype(np.float32)


# --------------------------------------------------------------------------
# features and weights
# --------------------------------------------------------------------------
def normal_matrix(seed: int, name: str, rows: int, cols: int, std: float) -> np.ndarray:
    st = Stream(seed, name)
    return (std * st.normal(rows * cols)).reshape(rows, cols).astype(np.float32)


def lifted_features(seed: int, raw: np.ndarray, channels: int) -> np.ndarray:
    """Lift raw per-point attributes (m x r) to `channels` by a fixed random
    r x channels matrix (input preparation, as for xyz+RGB or intensity)."""
    r = raw.shape[1]
    lift = normal_matrix(seed, "lift", r, channels, 1.0 / np.sqrt(r))
    return (raw.astype(np.float64) @ lift.astype(np.float64)).astype(np.float32)


def conv_weights(seed: int, name: str, taps: int, cin: int, cout: int, std: float | None = None) -> np.ndarray:
    """Weights of one lattice convolution, taps x cin x cout, N(0, std^2);
    std defaults to 1/sqrt(taps*cin)."""
    if std is None:
        std = 1.0 / np.sqrt(taps * cin)
    st = Stream(seed, "W:" + name)
    return (std * st.normal(taps * cin * cout)).reshape(taps, cin, cout).astype(np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns.  Used to store bf16 inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r = np.where(nan, np.uint64(0x7FC0), r)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)

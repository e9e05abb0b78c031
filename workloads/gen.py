"""Seeded generators: voxelised synthetic surfaces and random tensors.

Every workload ``i`` draws from ``numpy.random.default_rng`` streams spawned
from ``SeedSequence(20211107 + i)`` in a fixed order: geometry, features,
coefficients, upstream gradient, test transforms.

Voxelisation follows the paper's input rule (Sec. 4.1): a site is active when
its unit cell encloses at least one sampled surface point.  Points are sampled
densely (>= 32 per unit area) unless a workload asks for a fixed sparse count.
A shell-thickness knob ``tau`` offsets each dense sample along the surface
normal by U(-tau, tau) before voxelising.
"""
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

from .configs import WorkloadSpec, get_config

DENSITY = 32.0  # samples per unit^2 for dense surfaces


def _streams(spec: WorkloadSpec):
    ss = np.random.SeedSequence(spec.seed)
    geo, feat, coef, grad, xform = ss.spawn(5)
    return dict(geometry=geo, features=feat, coeffs=coef, grad=grad, transforms=xform)


def random_rotation(rng) -> np.ndarray:
    """Uniform random rotation from a normalised Gaussian quaternion."""
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


# ----------------------------------------------------------------------------
# surface samplers: return (points [n,3], normals [n,3]) in the local frame
# ----------------------------------------------------------------------------

def _unit_sphere(rng, n):
    u = rng.standard_normal((n, 3))
    return u / np.linalg.norm(u, axis=1, keepdims=True)


def ellipsoid_dense(rng, axes):
    a = np.sort(np.asarray(axes, float))
    n = int(np.ceil(DENSITY * 4 * np.pi * a[1] * a[2]))  # bounds the map's area stretch
    u = _unit_sphere(rng, n)
    p = u * axes
    nrm = u / axes
    return p, nrm / np.linalg.norm(nrm, axis=1, keepdims=True)


def ellipsoid_uniform(rng, axes, n):
    """Area-uniform points on an ellipsoid by rejection on the area element."""
    axes = np.asarray(axes, float)
    gmax = 1.0 / axes.min()
    out = []
    need = n
    while need > 0:
        u = _unit_sphere(rng, 4 * need + 64)
        g = np.sqrt(((u / axes) ** 2).sum(1))
        keep = rng.uniform(0, gmax, len(u)) < g
        out.append(u[keep][:need] * axes)
        need -= len(out[-1])
    return np.concatenate(out)[:n]


def _box_faces(h):
    faces = []
    for ax in range(3):
        o1, o2 = [a for a in range(3) if a != ax]
        for sgn in (-1.0, 1.0):
            faces.append((ax, sgn, o1, o2, 4.0 * h[o1] * h[o2]))
    return faces


def _box_points(rng, h, counts):
    pts, nrms = [], []
    for (ax, sgn, o1, o2, _), c in zip(_box_faces(h), counts):
        p = np.zeros((c, 3))
        p[:, ax] = sgn * h[ax]
        p[:, o1] = rng.uniform(-h[o1], h[o1], c)
        p[:, o2] = rng.uniform(-h[o2], h[o2], c)
        nr = np.zeros((c, 3))
        nr[:, ax] = sgn
        pts.append(p)
        nrms.append(nr)
    return np.concatenate(pts), np.concatenate(nrms)


def box_dense(rng, h):
    counts = [int(np.ceil(DENSITY * f[4])) for f in _box_faces(h)]
    return _box_points(rng, h, counts)


def box_uniform(rng, h, n):
    areas = np.array([f[4] for f in _box_faces(h)])
    counts = rng.multinomial(n, areas / areas.sum())
    return _box_points(rng, h, counts)[0]


def _cyl_parts(h):
    r, hh = 0.5 * (h[0] + h[1]), h[2]
    return r, hh, np.array([2 * np.pi * r * 2 * hh, np.pi * r * r, np.pi * r * r])


def _cyl_points(rng, h, counts):
    r, hh, _ = _cyl_parts(h)
    c0, c1, c2 = counts
    th = rng.uniform(0, 2 * np.pi, c0)
    side = np.stack([r * np.cos(th), r * np.sin(th), rng.uniform(-hh, hh, c0)], 1)
    side_n = np.stack([np.cos(th), np.sin(th), np.zeros(c0)], 1)
    caps, caps_n = [], []
    for c, z in ((c1, -hh), (c2, hh)):
        rr = r * np.sqrt(rng.uniform(0, 1, c))
        t = rng.uniform(0, 2 * np.pi, c)
        caps.append(np.stack([rr * np.cos(t), rr * np.sin(t), np.full(c, z)], 1))
        caps_n.append(np.tile([0.0, 0.0, np.sign(z)], (c, 1)))
    return np.concatenate([side] + caps), np.concatenate([side_n] + caps_n)


def cylinder_dense(rng, h):
    _, _, areas = _cyl_parts(h)
    return _cyl_points(rng, h, [int(np.ceil(DENSITY * a)) for a in areas])


def cylinder_uniform(rng, h, n):
    _, _, areas = _cyl_parts(h)
    return _cyl_points(rng, h, rng.multinomial(n, areas / areas.sum()))[0]


def _thicken(rng, p, nrm, tau):
    if tau > 0:
        p = p + nrm * rng.uniform(-tau, tau, (len(p), 1))
    return p


def voxelise(points: np.ndarray, grid: int, lo: int = 0, hi: Optional[int] = None) -> np.ndarray:
    """Unique integer cells [m,3] (lexicographic) enclosing the points, clipped to [lo, hi)."""
    hi = grid if hi is None else hi
    v = np.floor(points).astype(np.int64)
    keep = np.all((v >= lo) & (v < hi), axis=1)
    return np.unique(v[keep], axis=0)


def _with_batch(cells_per_obj: List[np.ndarray]) -> np.ndarray:
    rows = [np.concatenate([np.full((len(c), 1), b, np.int64), c], 1)
            for b, c in enumerate(cells_per_obj)]
    out = np.concatenate(rows) if rows else np.zeros((0, 4), np.int64)
    return np.unique(out, axis=0).astype(np.int32)


# ----------------------------------------------------------------------------
# geometry per workload
# ----------------------------------------------------------------------------

def _geometry(spec: WorkloadSpec, rng) -> np.ndarray:
    g, p = spec.grid, spec.params
    if spec.geometry == "sphere":
        c = np.full(3, g / 2.0) + rng.uniform(-1, 1, 3)
        pts, nrm = ellipsoid_dense(rng, np.full(3, p["radius"]))
        return _with_batch([voxelise(_thicken(rng, pts, nrm, p["tau"]) + c, g)])
    if spec.geometry in ("ellipsoids", "scene"):
        lo, hi = p["axes"]
        clo, chi = p["centre"]
        allpts = []
        for k in range(p["n"]):
            kind = "ellipsoid" if (spec.geometry == "ellipsoids" or k % 2 == 0) else "box"
            ext = rng.uniform(lo, hi, 3)
            R = random_rotation(rng)
            c = rng.uniform(clo, chi, 3)
            pts, nrm = ellipsoid_dense(rng, ext) if kind == "ellipsoid" else box_dense(rng, ext)
            allpts.append(_thicken(rng, pts, nrm, p["tau"]) @ R.T + c)
        return _with_batch([voxelise(np.concatenate(allpts), g)])
    if spec.geometry in ("objects_sparse", "objects_dense"):
        lo, hi = p["extent"]
        cells = []
        for _ in range(spec.batch):
            kind = rng.integers(0, 3)
            ext = rng.uniform(lo, hi, 3) * p.get("scale", 1.0)
            R = random_rotation(rng)
            c = 32.0 + rng.uniform(-4, 4, 3)
            if spec.geometry == "objects_sparse":
                n = p["n_points"]
                pts = (ellipsoid_uniform(rng, ext, n), box_uniform(rng, ext, n),
                       cylinder_uniform(rng, ext, n))[kind]
                cells.append(voxelise(pts @ R.T + c, g))
            else:
                pts, _ = (ellipsoid_dense, box_dense, cylinder_dense)[kind](rng, ext)
                m = p["margin"]
                cells.append(voxelise(pts @ R.T + c, g, lo=m, hi=g - m))
        return _with_batch(cells)
    raise ValueError(spec.geometry)


# ----------------------------------------------------------------------------
# public API
# ----------------------------------------------------------------------------

@dataclass
class Workload:
    spec: WorkloadSpec
    coords: np.ndarray          # int32 [N, 4] as (b, x, y, z), lexicographic
    feats: np.ndarray           # float32 [N, Cin of layer 0] (bf16-rounded for bf16 workloads)
    coeffs: List[np.ndarray]    # float32 per layer

    @property
    def n(self) -> int:
        return len(self.coords)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32."""
    b = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(np.shape(x))


def make_features(spec: WorkloadSpec, n: int, cin: int, rounded: bool = True) -> np.ndarray:
    """N(0, 1) features in fp32; rounded to bfloat16 for a bf16 workload unless rounded=False."""
    rng = np.random.default_rng(_streams(spec)["features"])
    f = rng.standard_normal((n, cin)).astype(np.float32)
    return round_bf16(f) if spec.dtype == "bf16" and rounded else f


def make_coeffs(spec: WorkloadSpec, counts: List[int]) -> List[np.ndarray]:
    """Basis coefficients per layer: N(0,1) for the 16^3 workload, else N(0, 1/fan_in), fan_in = Cin*|S|."""
    rng = np.random.default_rng(_streams(spec)["coeffs"])
    out = []
    for layer, c in zip(spec.layers, counts):
        std = 1.0 if spec.index == 1 else 1.0 / np.sqrt(layer.cin * layer.n_offsets)
        out.append((rng.standard_normal(c) * std).astype(np.float32))
    return out


def make_grad(spec: WorkloadSpec, n_out: int, cout: int) -> np.ndarray:
    """Upstream gradient N(0,1) [n_out, cout] for the last layer's output."""
    rng = np.random.default_rng(_streams(spec)["grad"])
    g = rng.standard_normal((n_out, cout)).astype(np.float32)
    return round_bf16(g) if spec.dtype == "bf16" else g


def transform_rng(spec: WorkloadSpec):
    return np.random.default_rng(_streams(spec)["transforms"])


def make_coords(spec: WorkloadSpec) -> np.ndarray:
    return _geometry(spec, np.random.default_rng(_streams(spec)["geometry"]))


def make_workload(i, coeff_counts: Optional[List[int]] = None) -> Workload:
    """Coordinates, layer-0 features and (if counts are given) per-layer coefficients."""
    spec = get_config(i) if not isinstance(i, WorkloadSpec) else i
    coords = make_coords(spec)
    feats = make_features(spec, len(coords), spec.layers[0].cin)
    coeffs = make_coeffs(spec, coeff_counts) if coeff_counts is not None else []
    return Workload(spec, coords, feats, coeffs)


def make_point_cloud(spec: WorkloadSpec):
    """Raw object point clouds (no voxelisation): (points float32 [n, 3] in voxel units, batch
    int32 [n], features float32 [n, 4] = (R, G, B, 1) with R, G, B ~ U(0, 1)).  Objects follow
    the sparse-object recipe (box / cylinder / ellipsoid, random rotation, centre 32 + U(-4, 4)^3)
    with params["n_points"] area-uniform points each; points are listed object by object."""
    rng = np.random.default_rng(_streams(spec)["geometry"])
    lo, hi = spec.params["extent"]
    n = spec.params["n_points"]
    pts, bat = [], []
    for b in range(spec.batch):
        kind = rng.integers(0, 3)
        ext = rng.uniform(lo, hi, 3)
        R = random_rotation(rng)
        c = 32.0 + rng.uniform(-4, 4, 3)
        p = (ellipsoid_uniform(rng, ext, n), box_uniform(rng, ext, n), cylinder_uniform(rng, ext, n))[kind]
        pts.append(p @ R.T + c)
        bat.append(np.full(len(p), b, np.int32))
    points = np.concatenate(pts).astype(np.float32)
    frng = np.random.default_rng(_streams(spec)["features"])
    rgb = frng.uniform(0.0, 1.0, (len(points), 3)).astype(np.float32)
    feats = np.concatenate([rgb, np.ones((len(points), 1), np.float32)], 1)
    return points, np.concatenate(bat), feats


def make_motion(spec: WorkloadSpec):
    """A seeded rigid motion (rotation R [3, 3], translation t [3]) that turns the grid about its
    centre (uniform random rotation) and shifts it by U(-2, 2) voxels per axis."""
    rng = transform_rng(spec)
    R = random_rotation(rng)
    c = np.full(3, spec.grid / 2.0)
    t = c - R @ c + rng.uniform(-2.0, 2.0, 3)
    return R, t


def make_query_points(spec: WorkloadSpec, coords: np.ndarray):
    """params["per_site"] points per site: its cell centre (x + 1/2, voxel units, origin 0) plus
    U(-1, 1) per axis; returns (points float32 [m, 3], batch int32 [m])."""
    rng = transform_rng(spec)
    k = spec.params["per_site"]
    c = np.repeat(np.asarray(coords, np.int64), k, axis=0)
    pts = (c[:, 1:] + 0.5 + rng.uniform(-1.0, 1.0, (len(c), 3))).astype(np.float32)
    return pts, c[:, 0].astype(np.int32)


def shuffle_rows(seed: int, n: int) -> np.ndarray:
    """A seeded permutation of n rows (used to test row-order independence)."""
    return np.random.default_rng(seed).permutation(n)

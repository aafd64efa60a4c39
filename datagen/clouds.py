"""Seeded synthetic stand-ins for the paper's evaluation clouds.

The paper evaluates on ShapeNet part segmentation (objects of about 2.6K
points, processed one at a time), ScanNet rooms (9K-537K points, whole room),
SemanticKITTI LiDAR scans (82K-129K points, no cropping) and a three-scan
motion-segmentation window (Sec. "Experiments", dataset paragraphs).  None of
those datasets is used here: every cloud below is generated from a seed with
the shape, size and density structure of one of those families.

Nothing in this module computes any part of the lattice method; it only
emits positions, features, optional batch ids and convolution weights.

Weight layout for a lattice convolution is out-channel major,
``[C_out][T][C_in]`` float32, with ``T = 2(d+1)+1`` taps.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np


@dataclass
class ConvSpec:
    c_in: int
    c_out: int
    dtype: str  # "f32" or "bf16"
    weight: np.ndarray  # float32 [C_out][T][C_in]


@dataclass
class Workload:
    name: str
    config: int
    d: int
    sigma: Tuple[float, ...]
    pos: np.ndarray  # float32 [m][d]
    feat: np.ndarray  # float32 [m][C]
    batch: Optional[np.ndarray] = None  # int32 [m] or None
    convs: List[ConvSpec] = field(default_factory=list)
    extra: dict = field(default_factory=dict)

    @property
    def m(self) -> int:
        return int(self.pos.shape[0])

    @property
    def C(self) -> int:
        return int(self.feat.shape[1])

    @property
    def taps(self) -> int:
        return 2 * (self.d + 1) + 1


CONFIGS = {
    1: "tiny: 4096 points on 3 spheres, d=3, sigma=0.05, C=8, conv 8->16 f32",
    2: "part-seg batch: 16 objects x 2500 points, d=3, sigma=0.04, C=64, conv 64->64 f32 and bf16",
    3: "indoor room: 200k points, d=3, sigma=0.04 m, C=64 (from 6 rgb+normal), conv 64->64 and 64->128 bf16",
    4: "lidar scan: ~1.1e5 points from a 64-beam sensor, d=3, sigma=0.3 m, C=128, conv 128->128 bf16",
    5: "spatio-temporal: 4 lidar frames, ~4.5e5 points in (x,y,z,0.5 t), d=4, sigma=0.3, C=64, conv 64->64 bf16",
}


# ----------------------------------------------------------------------------
# small geometric helpers (input generation only)
# ----------------------------------------------------------------------------

def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array(
        [
            [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
            [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
            [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
        ]
    )


def _yaw(theta: float) -> np.ndarray:
    c, s = np.cos(theta), np.sin(theta)
    return np.array([[c, -s, 0.0], [s, c, 0.0], [0.0, 0.0, 1.0]])


def _sample_box_surface(rng, half, n, faces=("+x", "-x", "+y", "-y", "+z", "-z")):
    """Uniform samples on the given faces of an axis-aligned box centred at 0.

    Returns (points [n,3], normals [n,3], face index [n])."""
    a, b, c = half
    area = {"+x": 4 * b * c, "-x": 4 * b * c, "+y": 4 * a * c, "-y": 4 * a * c,
            "+z": 4 * a * b, "-z": 4 * a * b}
    w = np.array([area[f] for f in faces], dtype=np.float64)
    which = rng.choice(len(faces), size=n, p=w / w.sum())
    u = rng.uniform(-1.0, 1.0, size=(n, 2))
    pts = np.empty((n, 3))
    nrm = np.zeros((n, 3))
    for fi, f in enumerate(faces):
        sel = which == fi
        k = int(sel.sum())
        if k == 0:
            continue
        axis = "xyz".index(f[1])
        sign = 1.0 if f[0] == "+" else -1.0
        others = [i for i in range(3) if i != axis]
        p = np.empty((k, 3))
        p[:, axis] = sign * half[axis]
        p[:, others[0]] = u[sel, 0] * half[others[0]]
        p[:, others[1]] = u[sel, 1] * half[others[1]]
        pts[sel] = p
        nrm[sel, axis] = sign
    return pts, nrm, which


def _sample_cylinder_surface(rng, r, h, n):
    side = 2 * np.pi * r * h
    cap = np.pi * r * r
    w = np.array([side, cap, cap])
    which = rng.choice(3, size=n, p=w / w.sum())
    th = rng.uniform(0, 2 * np.pi, size=n)
    pts = np.empty((n, 3))
    s = which == 0
    pts[s, 0] = r * np.cos(th[s])
    pts[s, 1] = r * np.sin(th[s])
    pts[s, 2] = rng.uniform(-h / 2, h / 2, size=int(s.sum()))
    for ci, z in ((1, h / 2), (2, -h / 2)):
        s = which == ci
        rad = r * np.sqrt(rng.uniform(0, 1, size=int(s.sum())))
        pts[s, 0] = rad * np.cos(th[s])
        pts[s, 1] = rad * np.sin(th[s])
        pts[s, 2] = z
    return pts


def _conv_weight(rng, c_in, c_out, taps, std=0.1):
    return (rng.standard_normal((c_out, taps, c_in)) * std).astype(np.float32)


# ----------------------------------------------------------------------------
# the five workloads
# ----------------------------------------------------------------------------

def _tiny(seed: int) -> Workload:
    rng = np.random.default_rng(seed)
    m = 4096
    r = rng.uniform(0.1, 0.3, size=3)
    centres = rng.uniform(r[:, None], 1.0 - r[:, None], size=(3, 3))
    area = 4 * np.pi * r * r
    counts = rng.multinomial(m, area / area.sum())
    pts = []
    for i in range(3):
        v = rng.standard_normal((counts[i], 3))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        pts.append(centres[i] + r[i] * v)
    pos = np.concatenate(pts)[rng.permutation(m)].astype(np.float32)
    feat = rng.standard_normal((m, 8)).astype(np.float32)
    convs = [ConvSpec(8, 16, "f32", _conv_weight(rng, 8, 16, 9))]
    return Workload("tiny-spheres", 1, 3, (0.05,) * 3, pos, feat, None, convs)


def _partseg(seed: int) -> Workload:
    rng = np.random.default_rng(seed)
    n_obj, per = 16, 2500
    all_pts, all_b = [], []
    for obj in range(n_obj):
        n_prim = int(rng.integers(2, 5))
        prims = []
        for _ in range(n_prim):
            if rng.random() < 0.5:
                half = rng.uniform(0.05, 0.5, size=3)
                area = 8 * (half[0] * half[1] + half[1] * half[2] + half[0] * half[2])
                prims.append(("box", half, area))
            else:
                rad = rng.uniform(0.05, 0.3)
                hgt = rng.uniform(0.1, 1.0)
                area = 2 * np.pi * rad * hgt + 2 * np.pi * rad * rad
                prims.append(("cyl", (rad, hgt), area))
        areas = np.array([p[2] for p in prims])
        counts = rng.multinomial(per, areas / areas.sum())
        pts = []
        for (kind, prm, _), k in zip(prims, counts):
            if kind == "box":
                p, _, _ = _sample_box_surface(rng, prm, int(k))
            else:
                p = _sample_cylinder_surface(rng, prm[0], prm[1], int(k))
            rot = _random_rotation(rng)
            centre = rng.uniform(-0.5, 0.5, size=3)
            pts.append(p @ rot.T + centre)
        p = np.concatenate(pts)
        p -= p.mean(axis=0)
        p /= np.linalg.norm(p, axis=1).max()
        all_pts.append(p)
        all_b.append(np.full(per, obj, dtype=np.int32))
    pos = np.concatenate(all_pts)
    batch = np.concatenate(all_b)
    perm = rng.permutation(pos.shape[0])
    pos = pos[perm].astype(np.float32)
    batch = batch[perm]
    feat = rng.standard_normal((pos.shape[0], 64)).astype(np.float32)
    convs = [ConvSpec(64, 64, "f32", _conv_weight(rng, 64, 64, 9)),
             ConvSpec(64, 64, "bf16", _conv_weight(rng, 64, 64, 9))]
    return Workload("partseg-batch16", 2, 3, (0.04,) * 3, pos, feat, batch, convs)


def _indoor(seed: int) -> Workload:
    rng = np.random.default_rng(seed)
    m = 200_000
    L, H = 8.0, 3.0
    # surfaces: (kind, params, area, colour)
    surfs = []
    surfs.append(("plane", dict(origin=np.zeros(3), u=np.array([L, 0, 0.]), v=np.array([0, L, 0.]),
                                n=np.array([0, 0, 1.])), L * L))
    for origin, u, n in (
        (np.array([0, 0, 0.]), np.array([0, L, 0.]), np.array([1, 0, 0.])),
        (np.array([L, 0, 0.]), np.array([0, L, 0.]), np.array([-1, 0, 0.])),
        (np.array([0, 0, 0.]), np.array([L, 0, 0.]), np.array([0, 1, 0.])),
        (np.array([0, L, 0.]), np.array([L, 0, 0.]), np.array([0, -1, 0.])),
    ):
        surfs.append(("plane", dict(origin=origin, u=u, v=np.array([0, 0, H]), n=n), L * H))
    for _ in range(20):
        half = np.array([rng.uniform(0.3, 2.0) / 2, rng.uniform(0.3, 2.0) / 2, rng.uniform(0.3, 1.5) / 2])
        yaw = rng.uniform(0, 2 * np.pi)
        centre = np.array([rng.uniform(1.0, L - 1.0), rng.uniform(1.0, L - 1.0), half[2]])
        a, b, c = half
        area = 4 * a * b + 2 * (4 * a * c) + 2 * (4 * b * c)
        surfs.append(("box", dict(half=half, yaw=yaw, centre=centre), area))
    areas = np.array([s[2] for s in surfs])
    counts = rng.multinomial(m, areas / areas.sum())
    colours = rng.uniform(0, 1, size=(len(surfs), 3))
    pts, nrms, cols = [], [], []
    for si, ((kind, prm, _), k) in enumerate(zip(surfs, counts)):
        k = int(k)
        if kind == "plane":
            uv = rng.uniform(0, 1, size=(k, 2))
            p = prm["origin"] + uv[:, :1] * prm["u"] + uv[:, 1:] * prm["v"]
            n = np.broadcast_to(prm["n"], (k, 3)).copy()
        else:
            p, n, _ = _sample_box_surface(rng, prm["half"], k, faces=("+x", "-x", "+y", "-y", "+z"))
            R = _yaw(prm["yaw"])
            p = p @ R.T + prm["centre"]
            n = n @ R.T
        p = p + n * rng.normal(0.0, 0.005, size=(k, 1))
        pts.append(p)
        nrms.append(n)
        cols.append(np.broadcast_to(colours[si], (k, 3)))
    pos = np.concatenate(pts)
    feat6 = np.concatenate([np.concatenate(cols), np.concatenate(nrms)], axis=1)
    perm = rng.permutation(m)
    pos = pos[perm].astype(np.float32)
    feat6 = feat6[perm].astype(np.float32)
    lift = rng.normal(0.0, np.sqrt(1.0 / 6.0), size=(6, 64))
    feat = (feat6.astype(np.float64) @ lift).astype(np.float32)
    convs = [ConvSpec(64, 64, "bf16", _conv_weight(rng, 64, 64, 9)),
             ConvSpec(64, 128, "bf16", _conv_weight(rng, 64, 128, 9))]
    return Workload("indoor-room", 3, 3, (0.04,) * 3, pos, feat, None, convs,
                    extra={"feat6": feat6})


def _lidar_scene(rng, n_boxes=40):
    boxes = []
    for _ in range(n_boxes):
        rad = np.sqrt(rng.uniform(3.0 ** 2, 45.0 ** 2))
        ang = rng.uniform(0, 2 * np.pi)
        size = np.array([rng.uniform(0.5, 6.0), rng.uniform(0.5, 3.0), rng.uniform(0.5, 3.0)])
        yaw = rng.uniform(0, 2 * np.pi)
        boxes.append(dict(centre=np.array([rad * np.cos(ang), rad * np.sin(ang), size[2] / 2]),
                          half=size / 2, yaw=yaw))
    return boxes


def _raycast(rng, boxes, n_beams=64, n_az=1875, origin=(0.0, 0.0, 1.73), max_range=50.0):
    """Return hit points in scan order (azimuth-major, beam-minor)."""
    o = np.array(origin)
    elev = np.deg2rad(np.linspace(-25.0, 3.0, n_beams))
    az = np.arange(n_az) * (2 * np.pi / n_az)
    A, E = np.meshgrid(az, elev, indexing="ij")  # [n_az, n_beams]
    dirs = np.stack([np.cos(E) * np.cos(A), np.cos(E) * np.sin(A), np.sin(E)], axis=-1).reshape(-1, 3)
    n = dirs.shape[0]
    t_best = np.full(n, np.inf)
    down = dirs[:, 2] < 0
    t_best[down] = -o[2] / dirs[down, 2]
    for b in boxes:
        R = _yaw(b["yaw"])
        lo_o = (o - b["centre"]) @ R  # into box frame
        ld = dirs @ R
        with np.errstate(divide="ignore", invalid="ignore"):
            inv = 1.0 / ld
            t1 = (-b["half"] - lo_o) * inv
            t2 = (b["half"] - lo_o) * inv
        tmin = np.nanmax(np.minimum(t1, t2), axis=1)
        tmax = np.nanmin(np.maximum(t1, t2), axis=1)
        hit = (tmax >= np.maximum(tmin, 0.0)) & (tmin > 0)
        t_best = np.where(hit & (tmin < t_best), tmin, t_best)
    keep = t_best <= max_range
    t = t_best[keep] + rng.normal(0.0, 0.02, size=int(keep.sum()))
    return o + t[:, None] * dirs[keep]


def _lidar(seed: int) -> Workload:
    rng = np.random.default_rng(seed)
    boxes = _lidar_scene(rng)
    pos = _raycast(rng, boxes).astype(np.float32)
    feat = rng.standard_normal((pos.shape[0], 128)).astype(np.float32)
    convs = [ConvSpec(128, 128, "bf16", _conv_weight(rng, 128, 128, 9))]
    return Workload("lidar-scan", 4, 3, (0.3,) * 3, pos, feat, None, convs)


def _spatiotemporal(seed: int) -> Workload:
    rng = np.random.default_rng(seed)
    boxes = _lidar_scene(rng)
    movers = rng.choice(len(boxes), size=10, replace=False)
    vel = {}
    for i in movers:
        speed = rng.uniform(0.0, 2.0)
        ang = rng.uniform(0, 2 * np.pi)
        vel[int(i)] = np.array([speed * np.cos(ang), speed * np.sin(ang), 0.0])
    frames = []
    for t in range(4):
        moved = []
        for i, b in enumerate(boxes):
            bb = dict(b)
            if i in vel:
                bb["centre"] = b["centre"] + t * vel[i]
            moved.append(bb)
        p = _raycast(rng, moved)
        frames.append(np.concatenate([p, np.full((p.shape[0], 1), 0.5 * t)], axis=1))
    pos = np.concatenate(frames).astype(np.float32)
    feat = rng.standard_normal((pos.shape[0], 64)).astype(np.float32)
    convs = [ConvSpec(64, 64, "bf16", _conv_weight(rng, 64, 64, 11))]
    return Workload("spatiotemporal-4frames", 5, 4, (0.3,) * 4, pos, feat, None, convs)


_GEN = {1: _tiny, 2: _partseg, 3: _indoor, 4: _lidar, 5: _spatiotemporal}


def make_workload(config: int) -> Workload:
    """Build workload ``config`` (1..5) from seed ``config``; deterministic."""
    return _GEN[config](config)


def random_cloud(m: int, d: int, seed: int, extent: float = 1.0, C: int = 4,
                 n_batch: int = 0) -> Workload:
    """Uniform random points in a cube, for small generic tests."""
    rng = np.random.default_rng(seed)
    pos = rng.uniform(-extent, extent, size=(m, d)).astype(np.float32)
    feat = rng.standard_normal((m, C)).astype(np.float32)
    batch = rng.integers(0, n_batch, size=m).astype(np.int32) if n_batch > 0 else None
    return Workload(f"random-{m}-{d}", 0, d, (1.0,) * d, pos, feat, batch, [])


def conv_weight(c_in: int, c_out: int, d: int, seed: int, std: float = 0.1) -> np.ndarray:
    """Seeded N(0, std^2) weights in ``[C_out][2(d+1)+1][C_in]`` layout."""
    return _conv_weight(np.random.default_rng(seed), c_in, c_out, 2 * (d + 1) + 1, std)


def random_rows(n: int, C: int, seed: int, std: float = 1.0) -> np.ndarray:
    """Seeded N(0, std^2) float32 rows [n, C]: stand-alone inputs for one stage
    (vertex values fed to a convolution or a slice)."""
    return (np.random.default_rng(seed).standard_normal((n, C)) * std).astype(np.float32)


# Output classes of the label sets each workload stands in for (50 part
# labels for part segmentation, 20 semantic classes for the indoor and the
# single-scan LiDAR benchmarks, 26 for the multi-scan one with moving
# classes); the tiny cloud takes 8.  Used only as the classifier's width.
N_CLASSES = {1: 8, 2: 50, 3: 20, 4: 20, 5: 26}


@dataclass
class DeformWeights:
    w_delta: np.ndarray  # float32 [C]: the offsets' linear layer
    b_delta: float       # its bias
    w_cls: np.ndarray    # float32 [n_cls][C]: the classifier
    b_cls: np.ndarray    # float32 [n_cls]


def deform_weights(C: int, n_cls: int, seed: int, gain: float = 3.0) -> DeformWeights:
    """Seeded weights for a DeformSlice + classifier layer on C-channel vertex
    values: w_delta ~ N(0, gain^2 / C) (so that the offsets' pre-activations
    of N(0,1) rows spread over tanh's curved range rather than saturating),
    b_delta ~ N(0, 0.25), w_cls ~ N(0, 1/C), b_cls ~ N(0, 0.01)."""
    rng = np.random.default_rng(seed)
    w_delta = (rng.standard_normal(C) * (gain / np.sqrt(C))).astype(np.float32)
    b_delta = float(np.float32(rng.standard_normal() * 0.5))
    w_cls = (rng.standard_normal((n_cls, C)) / np.sqrt(C)).astype(np.float32)
    b_cls = (rng.standard_normal(n_cls) * 0.1).astype(np.float32)
    return DeformWeights(w_delta, b_delta, w_cls, b_cls)


# The PointNet of the network's first layer (1x1 widths 16, 32, 64 in the
# paper's figure) and the raw per-point features it sees: the indoor room's
# rgb + normal (6), the first three channels of the other object clouds and
# one channel (a remission-like scalar) for the LiDAR clouds.
POINTNET_WIDTHS = (16, 32, 64)


def raw_point_features(w: Workload) -> np.ndarray:
    """Raw per-point features [m, f_d] float32 of a workload (see above)."""
    if "feat6" in w.extra:
        return np.ascontiguousarray(w.extra["feat6"], dtype=np.float32)
    k = 1 if w.config in (4, 5) else 3
    return np.ascontiguousarray(w.feat[:, :k], dtype=np.float32)


def pointnet_weights(k0: int, d: int, sigma: float, seed: int, widths=POINTNET_WIDTHS):
    """Seeded PointNet parameters: a list of (a, s, W, b) per block, float32.

    a ~ 1 + N(0, 0.1^2) and s ~ N(0, 0.1^2) per input channel (a group
    normalisation's affine), except that the first block scales the d
    position channels by 1/sigma (offsets from the local mean are of the
    order of the lattice scale); W ~ N(0, 2/K) (He), b ~ N(0, 0.01^2)."""
    rng = np.random.default_rng(seed)
    out = []
    k = k0
    for li, w_out in enumerate(widths):
        a = (1.0 + 0.1 * rng.standard_normal(k)).astype(np.float32)
        if li == 0:
            a[:d] = a[:d] / np.float32(sigma)
        s = (0.1 * rng.standard_normal(k)).astype(np.float32)
        W = (rng.standard_normal((w_out, k)) * np.sqrt(2.0 / k)).astype(np.float32)
        b = (0.01 * rng.standard_normal(w_out)).astype(np.float32)
        out.append((a, s, W, b))
        k = w_out
    return out


def pointnet_gn_weights(k0: int, seed: int, widths=POINTNET_WIDTHS):
    """Seeded PointNet parameters with group normalisation: a list of
    (gamma, beta, W, b) per block, float32.  gamma ~ 1 + N(0, 0.1^2), beta ~
    N(0, 0.1^2) per input channel, W ~ N(0, 2/K) (He), b ~ N(0, 0.01^2)."""
    rng = np.random.default_rng(seed)
    out = []
    k = k0
    for w_out in widths:
        gamma = (1.0 + 0.1 * rng.standard_normal(k)).astype(np.float32)
        beta = (0.1 * rng.standard_normal(k)).astype(np.float32)
        W = (rng.standard_normal((w_out, k)) * np.sqrt(2.0 / k)).astype(np.float32)
        b = (0.01 * rng.standard_normal(w_out)).astype(np.float32)
        out.append((gamma, beta, W, b))
        k = w_out
    return out

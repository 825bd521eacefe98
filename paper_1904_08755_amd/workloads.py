"""Seeded synthetic workloads for the generalized sparse convolution.

This module only draws inputs: integer coordinates, features, weights and
upstream gradients, with fixed seeds.  It holds none of the method's
arithmetic (no hashing, no output coordinates, no kernel maps, no
convolution), so the CPU oracle and the HIP path can both be fed from it
without sharing any of the computation they are checked on.

Coordinates are rows ``(b, x1, ..., xD)`` of int32 (batch index first, the
sparse-tensor COO layout of Sec. 3, Eq. 1, with the batch column moved to the
front).  Features are row-major ``N x C``.  Weights are ``K x C_in x C_out``
(one ``C_in x C_out`` matrix per kernel offset, the transpose of the paper's
``W_i`` of Sec. 3.1).

Scene generator.  The paper measures on indoor scans (ScanNet, S3DIS) at
2 cm and on 3D videos built from Synthia (Sec. 7).  None of those datasets is
available, so a synthetic room stands in for them: the six faces of an
8 x 6 x 3 m room plus 20 random axis-aligned boxes resting on the floor
(five faces each: top and four sides), surface points drawn uniformly with
density proportional to face area, isotropic Gaussian noise of 0.5 cm, then
voxelised by ``floor(p / voxel)`` and de-duplicated.  The 3D-video workload
uses three frames of the same room in which every box moves 5 cm per frame
along its own random horizontal direction, with points re-drawn per frame.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

ROOT_SEED = 190408755

# stream ids of the seed sequence
S_GEOM, S_FEAT, S_WEIGHT, S_GRAD = 0, 1, 2, 3


def rng_for(config_id: int, stream: int, *extra: int) -> np.random.Generator:
    """Generator for one (config, stream[, sub-stream]) triple."""
    return np.random.default_rng(
        np.random.SeedSequence(ROOT_SEED, spawn_key=(config_id, stream) + tuple(extra)))


# --------------------------------------------------------------------------- #
# bf16 helpers (round-to-nearest-even on the raw bits).  Both sides of a parity
# check receive the same rounded bits, so no rounding decision is duplicated.
# --------------------------------------------------------------------------- #
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    assert np.isfinite(a).all()
    u = a.view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    # finite inputs: u + 0x8000 stays below 2**32, so uint32 cannot wrap
    return ((u + np.uint32(0x7FFF) + lsb) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------- #
# geometry
# --------------------------------------------------------------------------- #
def _box_faces(x0, y0, a, b, c, top=True):
    """Five faces (top + 4 sides) of a box on the floor, as (origin, u, v)."""
    o = np.array([x0, y0, 0.0])
    faces = []
    if top:
        faces.append((o + [0, 0, c], np.array([a, 0, 0.0]), np.array([0, b, 0.0])))
    faces.append((o, np.array([0, b, 0.0]), np.array([0, 0, c])))                 # x = x0
    faces.append((o + [a, 0, 0], np.array([0, b, 0.0]), np.array([0, 0, c])))     # x = x0 + a
    faces.append((o, np.array([a, 0, 0.0]), np.array([0, 0, c])))                 # y = y0
    faces.append((o + [0, b, 0], np.array([a, 0, 0.0]), np.array([0, 0, c])))     # y = y0 + b
    return faces


def _room_faces(L, W, H):
    z = np.zeros(3)
    return [
        (z, np.array([L, 0, 0.0]), np.array([0, W, 0.0])),                # floor
        (np.array([0, 0, H]), np.array([L, 0, 0.0]), np.array([0, W, 0.0])),  # ceiling
        (z, np.array([0, W, 0.0]), np.array([0, 0, H])),                  # x = 0
        (np.array([L, 0, 0]), np.array([0, W, 0.0]), np.array([0, 0, H])),   # x = L
        (z, np.array([L, 0, 0.0]), np.array([0, 0, H])),                  # y = 0
        (np.array([0, W, 0]), np.array([L, 0, 0.0]), np.array([0, 0, H])),   # y = W
    ]


@dataclasses.dataclass
class SceneGeom:
    room: Tuple[float, float, float]
    boxes: np.ndarray        # n_boxes x 5: x0, y0, a, b, c
    dirs: np.ndarray         # n_boxes x 2 horizontal unit directions (3D-video motion)


def draw_scene(rng: np.random.Generator, scale: float = 1.0, n_boxes: int = 20) -> SceneGeom:
    L, W, H = 8.0 * scale, 6.0 * scale, 3.0 * scale
    lo, hi = 0.3 * scale, 1.5 * scale
    boxes = np.zeros((n_boxes, 5))
    for i in range(n_boxes):
        a, b, c = rng.uniform(lo, hi, size=3)
        x0 = rng.uniform(0.0, L - a)
        y0 = rng.uniform(0.0, W - b)
        boxes[i] = (x0, y0, a, b, c)
    ang = rng.uniform(0.0, 2 * np.pi, size=n_boxes)
    dirs = np.stack([np.cos(ang), np.sin(ang)], axis=1)
    return SceneGeom((L, W, H), boxes, dirs)


def sample_points(geom: SceneGeom, rng: np.random.Generator, n_points: int,
                  shift: float = 0.0, noise: float = 0.005) -> np.ndarray:
    """Area-proportional uniform surface samples plus isotropic noise (metres)."""
    faces = list(_room_faces(*geom.room))
    for (x0, y0, a, b, c), d in zip(geom.boxes, geom.dirs):
        faces += _box_faces(x0 + shift * d[0], y0 + shift * d[1], a, b, c)
    areas = np.array([np.linalg.norm(np.cross(u, v)) for _, u, v in faces])
    counts = rng.multinomial(n_points, areas / areas.sum())
    pts = []
    for (o, u, v), n in zip(faces, counts):
        if n == 0:
            continue
        st = rng.uniform(0.0, 1.0, size=(n, 2))
        pts.append(o[None, :] + st[:, :1] * u[None, :] + st[:, 1:] * v[None, :])
    p = np.concatenate(pts, axis=0)
    p += rng.normal(0.0, noise, size=p.shape)
    return p


def voxel_rows(p: np.ndarray, voxel: float, b: int, t: Optional[int] = None) -> np.ndarray:
    """Voxel rows of points stored as float32, at a voxel size stored as
    float32: floor of the exact quotient of those two values.  The quotient of
    two float32 numbers rounded to float64 lies within 2^-53 of it relative,
    while a quotient that is not an integer lies at least 2^-24 (relative to
    the integer) from the next one, so for indices below 2^29 the float64
    floor is the exact one."""
    p32 = np.asarray(p, dtype=np.float32).astype(np.float64)
    v = np.floor(p32 / float(np.float32(voxel))).astype(np.int64)
    cols = [np.full((len(v), 1), b, np.int64), v]
    if t is not None:
        cols.append(np.full((len(v), 1), t, np.int64))
    return np.concatenate(cols, axis=1)


def unique_rows(rows: np.ndarray) -> np.ndarray:
    """De-duplicate integer rows (lexicographic order of np.unique)."""
    u = np.unique(rows, axis=0)
    assert np.abs(u).max() < 2**30
    return np.ascontiguousarray(u.astype(np.int32))


# --------------------------------------------------------------------------- #
# workloads
# --------------------------------------------------------------------------- #
@dataclasses.dataclass
class Layer:
    """One convolution of a workload.

    kind: "subm" (output coordinates = input coordinates), "down" (strided,
    output coordinates derived from the input by the stride) or "up" (the
    transposed convolution back to the coordinates of the matching "down").
    region: "cube" (hypercube of side ``ksize``), "cross", "hybrid" or "spatial".
    """
    kind: str
    region: str
    ksize: int
    stride: int
    c_in: int
    c_out: int
    W: np.ndarray                      # K x c_in x c_out float32 (bf16-rounded when dtype == bf16)
    W_bits: Optional[np.ndarray] = None  # uint16 bf16 bits when dtype == bf16


@dataclasses.dataclass
class Workload:
    config_id: int
    name: str
    D: int
    dtype: str                     # "f32" or "bf16"
    coords: np.ndarray             # N x (1 + D) int32
    X: np.ndarray                  # N x C float32 (bf16-rounded values when dtype == bf16)
    X_bits: Optional[np.ndarray]
    layers: List[Layer]
    dY: np.ndarray                 # gradient w.r.t. the last layer's output (float32 values)
    dY_bits: Optional[np.ndarray]
    n_points: Sequence[int] = ()

    @property
    def n(self) -> int:
        return int(self.coords.shape[0])


def _region_size(region: str, ksize: int, D: int) -> int:
    if region == "cube":
        return ksize ** D
    if region == "cross":
        return 2 * D * ((ksize - 1) // 2) + 1
    if region == "hybrid":
        return ksize ** (D - 1) + 2
    if region == "spatial":
        return ksize ** (D - 1)
    raise ValueError(region)


def _weights(cid: int, idx: int, K: int, ci: int, co: int) -> np.ndarray:
    rng = rng_for(cid, S_WEIGHT, idx)
    return (rng.standard_normal((K, ci, co)) / np.sqrt(K * ci)).astype(np.float32)


def _as_dtype(a: np.ndarray, dtype: str):
    if dtype == "bf16":
        bits = f32_to_bf16_bits(a)
        return bf16_bits_to_f32(bits).reshape(a.shape), bits.reshape(a.shape)
    return np.ascontiguousarray(a, np.float32), None


CONFIG_NAMES = {
    0: "random64_c3to16_cube3",
    1: "scene2cm_b2_c32_cube3",
    2: "scene2cm_b4_down2_c32to64_up2_c64to32",
    3: "video4d_5cm_t3_c32_hybrid29",
    4: "scene2cm_b2_c256_cube3_bf16",
}

SCENE_POINTS_2CM = 161_000
SCENE_POINTS_5CM = 46_500


def scene_coords(cid: int, batch: int, scale: float, voxel: float, n_points: int,
                 frames: Optional[int] = None) -> Tuple[np.ndarray, List[int]]:
    rows, npts = [], []
    n = int(round(n_points * scale * scale))
    for b in range(batch):
        geom = draw_scene(rng_for(cid, S_GEOM, b), scale=scale)
        if frames is None:
            p = sample_points(geom, rng_for(cid, S_GEOM, b, 1), n)
            rows.append(voxel_rows(p, voxel, b))
        else:
            for t in range(frames):
                p = sample_points(geom, rng_for(cid, S_GEOM, b, 1 + t), n, shift=0.05 * scale * t)
                rows.append(voxel_rows(p, voxel, b, t))
        npts.append(n)
    return unique_rows(np.concatenate(rows, axis=0)), npts


def make_workload(cid: int, scale: float = 1.0, region: Optional[str] = None) -> Workload:
    """Workload ``cid`` (0..4).  ``scale`` < 1 shrinks the scene (room, boxes and
    point count) for quick checks while keeping its structure; it is ignored for
    workload 0, which is already small.  ``region`` replaces the region of the 3D
    video (workload 3): "cube" gives the full 3^4 tesseract (81 offsets) that the
    hybrid kernel of Sec. 5.1 is a cheaper stand-in for, "spatial" the 3^3 cube
    at zero time offset (27 offsets: every frame convolved on its own)."""
    dtype = "bf16" if cid == 4 else "f32"
    npts: List[int] = []
    if cid == 0:
        rng = rng_for(cid, S_GEOM)
        flat = rng.choice(64 ** 3, 2000, replace=False)
        x, y, z = np.unravel_index(flat, (64, 64, 64))
        coords = np.stack([np.zeros_like(x), x, y, z], axis=1).astype(np.int32)
        D = 3
        specs = [("subm", "cube", 3, 1, 3, 16)]
    elif cid in (1, 4):
        coords, npts = scene_coords(cid, 2, scale, 0.02, SCENE_POINTS_2CM)
        D = 3
        c = 32 if cid == 1 else 256
        specs = [("subm", "cube", 3, 1, c, c)]
    elif cid == 2:
        coords, npts = scene_coords(cid, 4, scale, 0.02, SCENE_POINTS_2CM)
        D = 3
        specs = [("down", "cube", 2, 2, 32, 64), ("up", "cube", 2, 2, 64, 32)]
    elif cid == 3:
        coords, npts = scene_coords(cid, 1, scale, 0.05, SCENE_POINTS_5CM, frames=3)
        D = 4
        specs = [("subm", region or "hybrid", 3, 1, 32, 32)]
    else:
        raise ValueError(cid)

    N = coords.shape[0]
    X, Xb = _as_dtype(rng_for(cid, S_FEAT).standard_normal((N, specs[0][4])).astype(np.float32), dtype)
    layers = []
    for i, (kind, region, ks, st, ci, co) in enumerate(specs):
        K = _region_size(region, ks, D)
        W, Wb = _as_dtype(_weights(cid, i, K, ci, co), dtype)
        layers.append(Layer(kind, region, ks, st, ci, co, W, Wb))
    # the last layer's output lives on the input coordinates except for a
    # single strided layer; no workload ends on a "down" layer.
    assert layers[-1].kind != "down"
    dY, dYb = _as_dtype(rng_for(cid, S_GRAD).standard_normal((N, layers[-1].c_out)).astype(np.float32), dtype)
    name = CONFIG_NAMES[cid]
    if region is not None and cid == 3 and region != "hybrid":
        name = f"video4d_5cm_t3_c32_{'tesseract' if region == 'cube' else region}{layers[0].W.shape[0]}"
    return Workload(cid, name, D, dtype, coords, X, Xb, layers, dY, dYb, npts)


def random_coords(seed: int, n: int, D: int, lo: int, hi: int, batch: int = 1) -> np.ndarray:
    """``n`` unique random rows (b, x1..xD) with b < batch and x in [lo, hi)."""
    rng = np.random.default_rng(np.random.SeedSequence(ROOT_SEED, spawn_key=(1000, seed)))
    span = hi - lo
    total = batch * span ** D
    n = min(n, total)
    flat = rng.choice(total, n, replace=False)
    idx = np.unravel_index(flat, (batch,) + (span,) * D)
    rows = np.stack(idx, axis=1).astype(np.int64)
    rows[:, 1:] += lo
    return rows.astype(np.int32)


def space_time_chroma_coords(seed: int, frames: int = 3, crops: int = 12, half: int = 16,
                             second_colour: float = 0.3) -> np.ndarray:
    """7D rows (b, x, y, z, t, r, g, b) at the extents the space-time-chroma
    convolution of Sec. 6 meets: the 2 cm voxels of an indoor scene seen in
    ``frames`` frames, and RGB colour channels of 0..255 each.

    To keep the row count small while the coordinates still span the whole
    scene, only the voxels within ``half`` voxels (per axis) of ``crops``
    centres are kept: the six voxels with the smallest and largest x, y and z
    (so the box is the full scene's) and random ones.  A voxel's colour is
    constant over cells of 8 x 8 x 8 voxels (a hash of the cell), so spatial
    and temporal neighbours often share it; a fraction ``second_colour`` of the
    voxels also holds a second colour, one channel off by one, so neighbours
    along the colour axes occur too."""
    rows, _ = scene_coords(2000 + seed, 1, 1.0, 0.02, SCENE_POINTS_2CM, frames=frames)
    rng = np.random.default_rng(np.random.SeedSequence(ROOT_SEED, spawn_key=(1003, seed)))
    xyz = rows[:, 1:4].astype(np.int64)
    centres = [int(xyz[:, a].argmin()) for a in range(3)] + [int(xyz[:, a].argmax()) for a in range(3)]
    centres += rng.choice(len(rows), max(crops - 6, 0), replace=False).tolist()
    keep = np.zeros(len(rows), bool)
    for i in centres:
        keep |= np.all(np.abs(xyz - xyz[i]) <= half, axis=1)
    r4 = rows[keep].astype(np.int64)
    cell = r4[:, 1:4] // 8
    h = (cell[:, 0] * 73856093) ^ (cell[:, 1] * 19349663) ^ (cell[:, 2] * 83492791)
    rgb = np.stack([(h >> s) & 255 for s in (0, 8, 16)], axis=1)
    r7 = np.concatenate([r4, rgb], axis=1)
    two = r7[rng.random(len(r7)) < second_colour].copy()
    ch = 5 + rng.integers(0, 3, len(two))
    at = np.arange(len(two))
    two[at, ch] = np.clip(two[at, ch] + rng.choice([-1, 1], len(two)), 0, 255)
    return unique_rows(np.concatenate([r7, two], axis=0).astype(np.int32))


def random_features(seed: int, n: int, c: int, dtype: str = "f32"):
    rng = np.random.default_rng(np.random.SeedSequence(ROOT_SEED, spawn_key=(1001, seed)))
    return _as_dtype(rng.standard_normal((n, c)).astype(np.float32), dtype)


def random_weights(seed: int, K: int, ci: int, co: int, dtype: str = "f32"):
    rng = np.random.default_rng(np.random.SeedSequence(ROOT_SEED, spawn_key=(1002, seed)))
    return _as_dtype((rng.standard_normal((K, ci, co)) / np.sqrt(K * ci)).astype(np.float32), dtype)

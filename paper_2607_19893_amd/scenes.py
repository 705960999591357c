"""Seeded synthetic inputs: scenes, cameras, target images and upstream gradients.

This module is the one piece of code shared by the HIP path's callers and the
CPU oracle's callers.  It draws numbers and builds pinhole cameras; it holds
none of the rendering, differentiation or optimisation arithmetic.  Everything
it returns is a plain numpy array (fp32 for anything the kernels consume).

The paper trains on MipNeRF360, Tanks & Temples, DeepBlending and MatrixCity
(Section 6.1, Table 2) but prints neither resolutions nor primitive counts, and
the datasets are not available here.  The five workloads below are seeded
synthetic stand-ins with the shapes of those captures: a tiny debug scene, an
object-centric ring capture, a forward-facing room-scale grid, a spiral
walk-through of a clustered scene, and one GPU's shard of a city-scale aerial
survey flown on a lawn-mower path.

Parameter conventions (per primitive, row-major, fp32):
  mean      [N,3]  world position
  log_scale [N,3]  log of the per-axis standard deviation
  quat      [N,4]  rotation quaternion (w, x, y, z), stored unit length
  opacity   [N]    opacity logit
  sh        [N,(L+1)^2,3]  spherical-harmonic colour coefficients, coefficient
                   k = l*l + l + m (m = -l..l), channel fastest

Camera convention: world-to-camera rotation R (rows = right, down, forward),
translation t = -R c, focal lengths from the horizontal field of view, the
principal point at the image centre, pixel (i, k) centred at (i+0.5, k+0.5).
Cameras are built in fp64 and rounded to fp32 once; both sides consume the
same fp32 numbers.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

TILE = 16
NEAR_Z = 0.2


@dataclasses.dataclass
class Camera:
    width: int
    height: int
    fx: float
    fy: float
    cx: float
    cy: float
    tan_fovx: float
    tan_fovy: float
    near_z: float
    R: np.ndarray        # (3,3) fp32, world -> camera
    t: np.ndarray        # (3,)  fp32
    campos: np.ndarray   # (3,)  fp32

    @property
    def tiles_x(self) -> int:
        return (self.width + TILE - 1) // TILE

    @property
    def tiles_y(self) -> int:
        return (self.height + TILE - 1) // TILE

    @property
    def num_tiles(self) -> int:
        return self.tiles_x * self.tiles_y


@dataclasses.dataclass
class Scene:
    mean: np.ndarray
    log_scale: np.ndarray
    quat: np.ndarray
    opacity: np.ndarray
    sh: np.ndarray
    sh_degree: int

    @property
    def n(self) -> int:
        return int(self.mean.shape[0])

    @property
    def sh_coeffs(self) -> int:
        return (self.sh_degree + 1) ** 2

    def permuted(self, perm) -> "Scene":
        """The same primitives stored in another order: row i of the result is row perm[i] of this scene."""
        perm = np.asarray(perm, np.int64)
        return Scene(mean=self.mean[perm], log_scale=self.log_scale[perm], quat=self.quat[perm],
                     opacity=self.opacity[perm], sh=self.sh[perm], sh_degree=self.sh_degree)

    def groups(self):
        """Parameter groups in the order used everywhere (name, array [N, cols])."""
        n = self.n
        return [("mean", self.mean.reshape(n, 3)),
                ("log_scale", self.log_scale.reshape(n, 3)),
                ("quat", self.quat.reshape(n, 4)),
                ("opacity", self.opacity.reshape(n, 1)),
                ("sh", self.sh.reshape(n, -1))]


@dataclasses.dataclass
class Workload:
    name: str
    scene: Scene
    cameras: List[Camera]
    seed: int
    target_kind: str      # "uniform", "smooth" or "perturbed"
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-15
    # storage order of the primitives: row i is row perm[i] of the generated
    # scene (None: the generator's order)
    perm: Optional[np.ndarray] = None

    def target_scene(self) -> "Scene":
        """The perturbed copy of the scene whose renders are the "perturbed"
        targets (the same physical scene whatever the storage order)."""
        return perturbed_copy(self.scene, self.seed, self.perm)

    def target(self, view: int, render=None) -> np.ndarray:
        """Target image [3,H,W] fp32 of a view.  "perturbed" targets are renders
        of target_scene() from the view's camera, made by the caller's
        render(scene, camera) (this module draws inputs and renders nothing)."""
        cam = self.cameras[view % len(self.cameras)]
        if self.target_kind == "perturbed":
            if render is None:
                raise ValueError("%s: targets are renders of the perturbed copy; pass render(scene, camera)"
                                 % self.name)
            if getattr(self, "_target_scene", None) is None:
                self._target_scene = self.target_scene()
            return np.ascontiguousarray(render(self._target_scene, cam), dtype=np.float32)
        return make_target(cam.width, cam.height, self.seed, view, self.target_kind)


def look_at(eye, target, up, width: int, height: int, fov_x_deg: float) -> Camera:
    """Pinhole camera at `eye` looking at `target`; fp64 construction, fp32 result."""
    eye = np.asarray(eye, np.float64)
    f = np.asarray(target, np.float64) - eye
    f /= np.linalg.norm(f)
    right = np.cross(f, np.asarray(up, np.float64))
    right /= np.linalg.norm(right)
    down = np.cross(f, right)
    R = np.stack([right, down, f])
    return _camera_from_pose(R, eye, width, height, fov_x_deg)


def look_along(eye, forward, up, width: int, height: int, fov_x_deg: float) -> Camera:
    eye = np.asarray(eye, np.float64)
    return look_at(eye, eye + np.asarray(forward, np.float64), up, width, height, fov_x_deg)


def _camera_from_pose(R, eye, width, height, fov_x_deg) -> Camera:
    tan_x = math.tan(math.radians(fov_x_deg) * 0.5)
    fx = width / (2.0 * tan_x)
    fy = fx
    tan_y = height / (2.0 * fy)
    t = -R @ eye
    f32 = np.float32
    return Camera(width=int(width), height=int(height), fx=float(f32(fx)), fy=float(f32(fy)),
                  cx=float(f32(width * 0.5)), cy=float(f32(height * 0.5)),
                  tan_fovx=float(f32(tan_x)), tan_fovy=float(f32(tan_y)), near_z=float(f32(NEAR_Z)),
                  R=R.astype(np.float32), t=t.astype(np.float32), campos=eye.astype(np.float32))


def normals(rng, shape, dtype=np.float32) -> np.ndarray:
    """Seeded standard normal samples of the given shape and dtype."""
    if dtype == np.float32:
        return rng.standard_normal(shape, dtype=np.float32)
    return rng.standard_normal(shape)


def random_quats(rng, n) -> np.ndarray:
    q = normals(rng, (n, 4), np.float64)
    q /= np.sqrt((q * q).sum(axis=1, keepdims=True))
    return q.astype(np.float32)


def _finish(rng, mean, ls_mu, ls_sd, logit_sd, logit_mu, degree, dc_kind) -> Scene:
    n = mean.shape[0]
    log_scale = normals(rng, (n, 3))
    log_scale *= np.float32(ls_sd)
    log_scale += np.float32(ls_mu)
    quat = random_quats(rng, n)
    opacity = normals(rng, (n,))
    opacity *= np.float32(logit_sd)
    opacity += np.float32(logit_mu)
    k = (degree + 1) ** 2
    # draw every coefficient N(0, 0.05) in place, then overwrite the DC term
    sh = np.empty((n, k, 3), np.float32)
    if k > 1:
        rng.standard_normal(dtype=np.float32, out=sh.reshape(-1))
        sh *= np.float32(0.05)
    if dc_kind == "rgb":
        # The colour itself is drawn U(0,1); the degree-0 coefficient that
        # yields it is (rgb - 0.5) / Y00 with the constant basis value
        # Y00 = 1 / (2 sqrt(pi)).
        rgb = rng.uniform(0.0, 1.0, (n, 3))
        sh[:, 0, :] = ((rgb - 0.5) * (2.0 * math.sqrt(math.pi))).astype(np.float32)
    else:
        sh[:, 0, :] = rng.random((n, 3), dtype=np.float32)
    return Scene(mean=np.ascontiguousarray(mean, dtype=np.float32), log_scale=log_scale, quat=quat,
                 opacity=opacity, sh=sh, sh_degree=degree)


def perturbed_copy(scene: "Scene", seed: int, perm: Optional[np.ndarray] = None) -> "Scene":
    """A seeded perturbation of a scene, the stand-in for the scene a set of
    photographs shows: means moved by N(0, 0.02) per axis, log-scales by
    N(0, 0.1), quaternion components by N(0, 0.05), opacity logits by N(0, 0.5)
    and every SH coefficient by N(0, 0.05).  The noise is drawn in the
    generator's order; perm (row i of `scene` is generated row perm[i]) picks
    each stored row's own noise."""
    rng = np.random.default_rng([seed, 4241])
    n = scene.n
    f32 = np.float32
    pick = (lambda a: a) if perm is None else (lambda a: a[perm])
    noise = [normals(rng, (n, 3)), normals(rng, (n, 3)), normals(rng, (n, 4)), normals(rng, scene.opacity.shape),
             normals(rng, scene.sh.shape)]
    return Scene(mean=(scene.mean + pick(noise[0]) * f32(0.02)).astype(f32),
                 log_scale=(scene.log_scale + pick(noise[1]) * f32(0.1)).astype(f32),
                 quat=(scene.quat + pick(noise[2]) * f32(0.05)).astype(f32),
                 opacity=(scene.opacity + pick(noise[3]) * f32(0.5)).astype(f32),
                 sh=(scene.sh + pick(noise[4]) * f32(0.05)).astype(f32),
                 sh_degree=scene.sh_degree)


def make_target(width: int, height: int, seed: int, view: int, kind: str) -> np.ndarray:
    """Target image [3,H,W] in [0,1].

    "uniform": i.i.d. U(0,1) per pixel.  "smooth": a seeded low-frequency
    colour field (four random plane waves per channel, built separably) plus
    +-5% uniform noise; it stands in for a photograph of the scene.
    """
    rng = np.random.default_rng([seed, 7919, view])
    if kind == "uniform":
        return rng.random((3, height, width), dtype=np.float32)
    ys = ((np.arange(height, dtype=np.float64) + 0.5) / height)[:, None]
    xs = ((np.arange(width, dtype=np.float64) + 0.5) / width)[None, :]
    img = np.empty((3, height, width), np.float32)
    for ch in range(3):
        acc = np.zeros((height, width), np.float32)
        for _ in range(4):
            fx_, fy_ = rng.uniform(-3.0, 3.0, 2)
            ph = rng.uniform(0, 2 * math.pi)
            ax = 2 * math.pi * fx_ * xs + ph
            by = 2 * math.pi * fy_ * ys
            # cos(a + b) = cos a cos b - sin a sin b, as two outer products
            acc += (np.cos(by) * np.cos(ax) - np.sin(by) * np.sin(ax)).astype(np.float32)
        noise = rng.random((height, width), dtype=np.float32)
        acc *= np.float32(0.1)
        acc += np.float32(0.45)
        acc += np.float32(0.1) * noise
        np.clip(acc, 0.0, 1.0, out=acc)
        img[ch] = acc
    return img


def make_upstream_grad(width: int, height: int, seed: int) -> np.ndarray:
    """A continuous upstream image gradient [3,H,W] of loss-like scale."""
    rng = np.random.default_rng([seed, 104729])
    scale = 2.0 / (3.0 * width * height)
    return ((rng.uniform(0.0, 1.0, (3, height, width)) - 0.5) * scale).astype(np.float32)


# --------------------------------------------------------------------------
# The five workloads.
# --------------------------------------------------------------------------

def tiny(seed: int = 0, n: int = 10_000) -> Workload:
    """10k Gaussians, SH degree 0, one 256x256 camera at (0,0,-4) looking +z."""
    rng = np.random.default_rng(seed)
    mean = rng.uniform(-1.0, 1.0, (n, 3))
    scene = _finish(rng, mean, -4.0, 0.5, 1.0, 0.0, 0, "rgb")
    cam = look_at((0.0, 0.0, -4.0), (0.0, 0.0, 0.0), (0.0, -1.0, 0.0), 256, 256, 60.0)
    return Workload("tiny-10k-L0-256px", scene, [cam], seed, "uniform")


def ring(seed: int = 1, n: int = 200_000, width: int = 1280, height: int = 720) -> Workload:
    """200k Gaussians in 20 isotropic clusters, SH degree 3, 8 cameras on a ring."""
    rng = np.random.default_rng(seed)
    centres = rng.uniform(-3.0, 3.0, (20, 3))
    which = rng.integers(0, 20, n)
    mean = centres[which] + 0.3 * normals(rng, (n, 3), np.float64)
    scene = _finish(rng, mean, -4.5, 0.7, 1.5, 0.0, 3, "coef")
    cams = []
    for i in range(8):
        th = 2 * math.pi * i / 8
        eye = (6.0 * math.cos(th), 0.0, 6.0 * math.sin(th))
        cams.append(look_at(eye, (0.0, 0.0, 0.0), (0.0, -1.0, 0.0), width, height, 60.0))
    return Workload("ring-200k-L3-720p", scene, cams, seed, "perturbed")


def room(seed: int = 2, n: int = 1_000_000, width: int = 1920, height: int = 1080) -> Workload:
    """1M Gaussians: 70% uniform in a 20x20x5 box, 30% in 50 clusters; 4x8 camera grid."""
    rng = np.random.default_rng(seed)
    n_uni = int(round(0.7 * n))
    lo = np.array([-10.0, -10.0, 0.0]); hi = np.array([10.0, 10.0, 5.0])
    uni = rng.uniform(lo, hi, (n_uni, 3))
    centres = rng.uniform(lo, hi, (50, 3))
    which = rng.integers(0, 50, n - n_uni)
    clu = centres[which] + 0.25 * normals(rng, (n - n_uni, 3), np.float64)
    mean = np.concatenate([uni, clu], axis=0)
    scene = _finish(rng, mean, -5.0, 0.8, 1.5, 0.0, 3, "coef")
    cams = []
    for y in (-8.0, -6.0, -4.0, -2.0):
        for x in np.linspace(-8.75, 8.75, 8):
            cams.append(look_along((x, y, 2.5), (0.0, 1.0, 0.0), (0.0, 0.0, 1.0), width, height, 70.0))
    return Workload("room-1M-L3-1080p", scene, cams, seed, "smooth")


def spiral(seed: int = 3, n: int = 3_000_000, width: int = 1600, height: int = 1063) -> Workload:
    """3M Gaussians in 200 anisotropic clusters; 64 cameras on a 2-turn spiral."""
    rng = np.random.default_rng(seed)
    k = 200
    centres = rng.uniform([-30.0, -30.0, 0.0], [30.0, 30.0, 10.0], (k, 3))
    rots = np.stack([_rand_rot(rng) for _ in range(k)])
    lam = rng.uniform(0.05, 2.0, (k, 3))
    which = rng.integers(0, k, n)
    z = normals(rng, (n, 3), np.float64) * np.sqrt(lam[which])
    mean = centres[which] + np.einsum("nij,nj->ni", rots[which], z)
    scene = _finish(rng, mean, -5.5, 1.0, 2.0, -0.5, 3, "coef")
    cams = []
    for i in range(64):
        s = i / 63.0
        phi = 4 * math.pi * s
        r = 20.0 - 15.0 * s
        eye = (r * math.cos(phi), r * math.sin(phi), 5.0)
        # tangent of the spiral (d eye / ds), horizontal
        dx = -15.0 * math.cos(phi) - r * 4 * math.pi * math.sin(phi)
        dy = -15.0 * math.sin(phi) + r * 4 * math.pi * math.cos(phi)
        cams.append(look_along(eye, (dx, dy, 0.0), (0.0, 0.0, 1.0), width, height, 65.0))
    return Workload("spiral-3M-L3-1600x1063", scene, cams, seed, "smooth")


def aerial(seed: int = 4, n: int = 10_000_000, width: int = 1920, height: int = 1080) -> Workload:
    """One GPU's shard of an aerial city scene: 10M Gaussians, lawn-mower path of 128 cameras."""
    rng = np.random.default_rng(seed)
    mean = np.empty((n, 3), np.float32)
    mean[:, 0] = rng.random(n, dtype=np.float32) * np.float32(1000.0) - np.float32(500.0)
    mean[:, 1] = rng.random(n, dtype=np.float32) * np.float32(1000.0) - np.float32(500.0)
    mean[:, 2] = np.abs(normals(rng, (n,)) * np.float32(20.0))
    scene = _finish(rng, mean, -3.0, 1.2, 2.0, 0.0, 3, "coef")
    cams = []
    c45 = math.cos(math.radians(45.0))
    for strip in range(8):
        y = -437.5 + 125.0 * strip
        xs = [-412.5 + 55.0 * j for j in range(16)]
        heading = 1.0
        if strip % 2 == 1:
            xs = xs[::-1]
            heading = -1.0
        for x in xs:
            fwd = (heading * c45, 0.0, -c45)
            cams.append(look_along((x, y, 150.0), fwd, (0.0, 0.0, 1.0), width, height, 60.0))
    return Workload("aerial-10M-L3-1080p", scene, cams, seed, "smooth")


def _rand_rot(rng) -> np.ndarray:
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - w * z), 2 * (x * z + w * y)],
                     [2 * (x * y + w * z), 1 - 2 * (x * x + z * z), 2 * (y * z - w * x)],
                     [2 * (x * z - w * y), 2 * (y * z + w * x), 1 - 2 * (x * x + y * y)]])


WORKLOADS = {"tiny": tiny, "ring": ring, "room": room, "spiral": spiral, "aerial": aerial}


def workload(name: str, **kw) -> Workload:
    return WORKLOADS[name](**kw)


def _spread7_table() -> np.ndarray:
    """For every 7-bit value, its bits moved to bits 0, 3, ..., 18."""
    t = np.zeros(128, np.uint64)
    for v in range(128):
        t[v] = sum(((v >> b) & 1) << (3 * b) for b in range(7))
    return t


_SPREAD7 = _spread7_table()


def _spread3(v: np.ndarray) -> np.ndarray:
    """Bits 0..20 of v moved to bits 0, 3, 6, ..., 60 (uint64), seven bits at a time."""
    v = np.asarray(v, np.uint32)
    out = _SPREAD7[v & 127]
    out |= _SPREAD7[(v >> 7) & 127] << np.uint64(21)
    out |= _SPREAD7[(v >> 14) & 127] << np.uint64(42)
    return out


def morton_codes(mean: np.ndarray, bits: int = 21) -> np.ndarray:
    """Z-order (Morton) code of each position: the coordinates quantized to
    `bits` bits (at most 21) over the points' bounding box, interleaved x, y, z
    from the lowest bit up."""
    m = np.asarray(mean, np.float32).reshape(-1, 3)
    if m.shape[0] == 0:
        return np.zeros(0, np.uint64)
    lo, hi = m.min(axis=0).astype(np.float64), m.max(axis=0).astype(np.float64)
    span = np.where(hi > lo, hi - lo, 1.0)
    code = np.zeros(m.shape[0], np.uint64)
    for k in range(3):
        q = ((m[:, k] - np.float32(lo[k])) * np.float32((2 ** bits - 1) / span[k])).astype(np.int64)
        q = np.clip(q, 0, 2 ** bits - 1).astype(np.uint32)
        code |= _spread3(q) << np.uint64(k)
    return code


def spatial_order(mean: np.ndarray) -> np.ndarray:
    """The storage order that places primitives near each other in space near
    each other in memory: ascending Morton code of the mean (equal codes keep
    their given order).  A view's visible set, a region of space, then falls
    into a few long runs of ids, so every per-primitive gather of the training
    view reads mostly whole, consecutive cache lines."""
    return np.argsort(morton_codes(mean), kind="stable")


def spatially_ordered(w: Workload) -> Workload:
    """The workload with its primitives stored in spatial order (same cameras, targets and content)."""
    p = spatial_order(w.scene.mean)
    return dataclasses.replace(w, scene=w.scene.permuted(p), perm=p if w.perm is None else w.perm[p])


def random_scene(seed: int, n: int, degree: int, extent: float = 1.0, ls_mu: float = -2.5,
                 ls_sd: float = 0.3, depth: float = 4.0) -> Scene:
    """Small scenes for unit tests: means in a box in front of a camera at the origin."""
    rng = np.random.default_rng(seed)
    mean = rng.uniform(-extent, extent, (n, 3))
    mean[:, 2] += depth
    return _finish(rng, mean, ls_mu, ls_sd, 1.0, 0.5, degree, "coef" if degree > 0 else "rgb")


def adam_state(seed: int, n: int, cols: int, scale_m: float = 1e-4, scale_v: float = 1e-8):
    """Non-zero first/second moments so that a step is not the degenerate first one."""
    rng = np.random.default_rng([seed, 31337, cols])
    m = (rng.standard_normal((n, cols)) * scale_m).astype(np.float32)
    v = (np.abs(rng.standard_normal((n, cols))) * scale_v).astype(np.float32)
    return m, v


@dataclasses.dataclass
class Capture:
    """Camera centres and feature tracks of a synthetic image capture.

    item_ptr / item_tracks are a CSR list of each image's track ids
    (ascending, no repeats); position holds the camera centres [n, 3]."""
    name: str
    position: np.ndarray       # [n, 3] float64
    item_ptr: np.ndarray       # [n + 1] int64
    item_tracks: np.ndarray    # int32
    n_tracks: int

    @property
    def n(self) -> int:
        return int(self.position.shape[0])

    def tracks_of(self, i: int) -> np.ndarray:
        return self.item_tracks[self.item_ptr[i]:self.item_ptr[i + 1]]


def capture_tracks(n_images: int, seed: int = 5, obs_per_image: float = 300.0, long_frac: float = 0.01,
                   spacing: float = 10.0, altitude: float = 120.0) -> Capture:
    """Stand-in for the SfM tracks of an aerial survey (the paper's planner
    input; no SfM reconstruction is available here).  Images sit on a
    lawn-mower flight grid (ids follow the flight path, every other row
    reversed) with jittered centres.  A track is a scene point seen by the
    images of an a x b block of neighbouring grid cells, a, b in 1..3
    (lengths 1-9, mean 4); a fraction ``long_frac`` of tracks are outliers
    seen by blocks of 8-20 cells a side (the long tracks an outlier cap
    removes).  About ``obs_per_image`` observations per image."""
    rng = np.random.default_rng(seed)
    n = int(n_images)
    side = max(1, int(math.ceil(math.sqrt(n))))
    rows = -(-n // side)
    # grid cell -> image id along the flight path (cells past n are empty)
    gy, gx = np.divmod(np.arange(rows * side), side)
    path_x = np.where(gy % 2 == 0, gx, side - 1 - gx)
    cell_id = np.full(rows * side, -1, np.int64)
    flat = gy * side + path_x
    cell_id[flat] = np.arange(rows * side)
    cell_id[cell_id >= n] = -1
    pos = np.zeros((n, 3))
    ids = cell_id[cell_id >= 0]
    cells = np.nonzero(cell_id >= 0)[0]
    pos[ids, 0] = (cells % side) * spacing + rng.normal(0.0, 0.1 * spacing, ids.size)
    pos[ids, 1] = (cells // side) * spacing + rng.normal(0.0, 0.1 * spacing, ids.size)
    pos[ids, 2] = altitude + rng.normal(0.0, 0.02 * altitude, ids.size)
    n_tracks = max(1, int(n * obs_per_image / 4.0))
    a = rng.integers(1, 4, n_tracks)
    b = rng.integers(1, 4, n_tracks)
    big = rng.random(n_tracks) < long_frac
    a[big] = rng.integers(8, 21, int(big.sum()))
    b[big] = rng.integers(8, 21, int(big.sum()))
    x0 = rng.integers(0, side, n_tracks)
    y0 = rng.integers(0, rows, n_tracks)
    cnt = a * b
    tr = np.repeat(np.arange(n_tracks), cnt)
    local = np.arange(int(cnt.sum())) - np.repeat(np.cumsum(cnt) - cnt, cnt)
    cx = np.repeat(x0, cnt) + local % np.repeat(a, cnt)
    cy = np.repeat(y0, cnt) + local // np.repeat(a, cnt)
    ok = (cx < side) & (cy < rows)
    img = np.full(tr.size, -1, np.int64)
    img[ok] = cell_id[cy[ok] * side + cx[ok]]
    ok = img >= 0
    img, tr = img[ok], tr[ok]
    o = np.argsort(img, kind="stable")       # track ids were generated ascending
    img, tr = img[o], tr[o]
    ptr = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(img, minlength=n), out=ptr[1:])
    return Capture("aerial-%d" % n, pos, ptr, tr.astype(np.int32), n_tracks)

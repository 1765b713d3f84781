"""Seeded synthetic inputs for the cached SqueezeNeRF renderer.

This module only *makes inputs*: camera poses, intrinsics and the four cache
arrays (three position sub-caches and the direction cache).  It holds none of
the rendering arithmetic, so both the HIP path and the CPU oracle can consume
what it produces without sharing any of the method's code.

Cache layout (SqueezeNeRF Sec. 3.3, "Caching"): for each ordered pair
j in {(x,y), (y,z), (z,x)} one dense n_p x n_p grid over the scene box holds
sigma^j (1 value) and u^j, v^j, w^j (D values each), i.e. 3D+1 values per
texel; the direction cache holds D values (beta) on an n_theta x n_phi grid.
The alternative decoder ("SqueezeNeRF (alt)", Sec. 3.2 Eq. 5) stores D_sigma
values of sigma^j per texel instead (3D + D_sigma values) and a linear map.

Array shapes produced here (the logical layout the C ABI accepts):
  sigma[j] : [n_p][n_p]        plane j indexed [first axis][second axis]
             ([n_p][n_p][D_sigma] for the linear decoder)
  uvw[j]   : [n_p][n_p][3D]    record = u[0..D) v[0..D) w[0..D)
  beta     : [n_theta][n_phi][D]
  poses    : [B][3][4] float32 camera-to-world [R | c], camera looks down -z

Synthetic density: a sum of isotropic Gaussian blobs baked per plane.  A 3-D
isotropic Gaussian factorises exactly into three planar Gaussians with twice
the variance (exp(-|d|^2/2s^2) = prod_j exp(-(da^2+db^2)/4s^2)), so one blob
is represented exactly by the product rule of Eq. 4; each planar factor is
cut to exactly zero beyond a planar radius rho_b so that empty space is
exactly empty.  The uvw components and beta are uniform in [-1, 1].
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

BOX_MIN = (-1.5, -1.5, -1.5)
BOX_MAX = (1.5, 1.5, 1.5)
NEAR = 2.0
FAR = 6.0

# plane j -> (first axis, second axis), in the order xy, yz, zx
PLANE_AXES = ((0, 1), (1, 2), (2, 0))


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic workload: image, sampling and cache shape."""
    name: str
    number: int              # seeds are derived from it (1000+n, 2000+n, ...)
    width: int
    height: int
    n_samples: int
    n_p: int
    D: int
    n_theta: int
    n_phi: int
    dtype: str               # "f32" or "f16" storage for sigma, uvw and beta
    n_blobs: int
    sigma_max: float
    r_min: float
    r_max: float
    n_poses: int = 1
    stratified: bool = False
    t_eps: float = 1e-4
    focal: Optional[float] = None  # default 1.25 * width
    sigma_channels: int = 0        # 0: Eq. 4 product of scalar sigma^j; > 0: Eq. 5 linear map
    forward: bool = False          # forward-facing capture marched in NDC (LLFF-shaped)
    sigma_dtype: Optional[str] = None  # storage of sigma^j if it differs from dtype

    @property
    def fx(self) -> float:
        return float(self.focal if self.focal is not None else 1.25 * self.width)

    @property
    def nominal_samples(self) -> int:
        """Samples per call: one ray per pixel, N samples per ray, B views."""
        return self.width * self.height * self.n_samples * self.n_poses


CONFIGS = {
    # 64x64, N=64, k=64, D=8, all fp32, direction cache 32x32
    "tiny": Config("tiny", 1, 64, 64, 64, 64, 8, 32, 32, "f32", 16, 50.0, 0.1, 0.4,
                   focal=80.0),
    # 800x800, N=192, k=256, D=8, fp16, direction cache 128x128
    "paper": Config("paper", 2, 800, 800, 192, 256, 8, 128, 128, "f16", 64, 50.0, 0.1, 0.4),
    # as "paper" with k=1024, direction cache 384x384, denser blobs
    "large": Config("large", 3, 800, 800, 192, 1024, 8, 384, 384, "f16", 64, 200.0, 0.1, 0.4),
    # 100 views on a spiral, caches as "paper"
    "batch": Config("batch", 4, 800, 800, 192, 256, 8, 128, 128, "f16", 64, 50.0, 0.1, 0.4,
                    n_poses=100),
    # 1920x1080, N=384 stratified, k=2048, D=16, direction cache 512x512
    "stress": Config("stress", 5, 1920, 1080, 384, 2048, 16, 512, 512, "f16", 256, 50.0,
                     0.02, 0.5, stratified=True),
    # as "tiny" with the Eq. 5 decoder (D_sigma = 12) and 48 blobs
    "tiny_alt": Config("tiny_alt", 8, 64, 64, 64, 64, 8, 32, 32, "f32", 48, 50.0, 0.1, 0.4,
                       focal=80.0, sigma_channels=12),
    # "SqueezeNeRF (alt)" decoder (Eq. 5, D_sigma = 12) on the paper shape
    "alt": Config("alt", 6, 800, 800, 192, 256, 8, 128, 128, "f16", 64, 50.0, 0.1, 0.4,
                  sigma_channels=12),
    # forward-facing (LLFF-shaped): 504x378, the paper's 512 cache with its
    # precisions (sigma fp32, uvw and beta fp16), n_d = 32, 256 samples in NDC
    "llff": Config("llff", 9, 504, 378, 256, 512, 8, 32, 32, "f16", 64, 50.0, 0.05, 0.25,
                   focal=0.8 * 504, forward=True, sigma_dtype="f32"),
    # a small forward-facing case the oracle renders in full
    "llff_tiny": Config("llff_tiny", 10, 48, 36, 64, 64, 8, 16, 16, "f32", 48, 50.0, 0.05, 0.25,
                        focal=0.8 * 48, forward=True),
    # the paper's own shape for its 800x800 timings: 256 samples per ray and
    # the 512 cache with its precisions (sigma fp32, uvw and beta fp16,
    # n_d = 64, D = 8), blobs as "paper"
    "paper512": Config("paper512", 11, 800, 800, 256, 512, 8, 64, 64, "f16", 64, 50.0, 0.1, 0.4,
                       sigma_dtype="f32"),
    # the alt decoder at the paper's alt cache size (n_p = 512, n_d = 256)
    "alt512": Config("alt512", 7, 800, 800, 192, 512, 8, 256, 256, "f16", 64, 50.0, 0.1, 0.4,
                     sigma_channels=12),
}


def look_at_pose(radius: float, azimuth_deg: float, elevation_deg: float) -> np.ndarray:
    """Camera-to-world [R | c] (float32, 3x4) for a camera on a sphere around
    the origin looking at it, world up = +z; camera axes: +x right, +y up,
    looking down -z."""
    az = math.radians(azimuth_deg)
    el = math.radians(elevation_deg)
    c = np.array([radius * math.cos(el) * math.cos(az),
                  radius * math.cos(el) * math.sin(az),
                  radius * math.sin(el)], dtype=np.float64)
    fwd = -c / np.linalg.norm(c)
    right = np.cross(fwd, np.array([0.0, 0.0, 1.0]))
    right /= np.linalg.norm(right)
    up = np.cross(right, fwd)
    pose = np.zeros((3, 4), dtype=np.float64)
    pose[:, 0] = right
    pose[:, 1] = up
    pose[:, 2] = -fwd
    pose[:, 3] = c
    return pose.astype(np.float32)


def single_pose() -> np.ndarray:
    """The one view of the single-camera workloads: radius 4, azimuth 45 deg,
    elevation 30 deg."""
    return look_at_pose(4.0, 45.0, 30.0)[None]


def spiral_poses(n: int, seed: int = 5000) -> np.ndarray:
    """n views on a seeded spiral: radius 3.5..4.5, elevation -30..30 deg."""
    rng = np.random.Generator(np.random.PCG64(seed))
    a0 = rng.uniform(0.0, 2.0 * math.pi)
    out = np.zeros((n, 3, 4), dtype=np.float32)
    for k in range(n):
        s = k / (n - 1) if n > 1 else 0.0
        r = 4.0 + 0.5 * math.cos(6.0 * math.pi * s)
        el = 30.0 * math.sin(2.0 * math.pi * s)
        az = math.degrees(a0 + 4.0 * math.pi * s)
        out[k] = look_at_pose(r, az, el)
    return out


@dataclasses.dataclass
class Blobs:
    centre: np.ndarray   # [n][3]
    radius: np.ndarray   # [n]
    sigma_max: float


def make_blobs(n: int, sigma_max: float, r_min: float, r_max: float, seed: int) -> Blobs:
    rng = np.random.Generator(np.random.PCG64(seed))
    centre = rng.uniform(-1.0, 1.0, size=(n, 3))
    radius = rng.uniform(r_min, r_max, size=n)
    return Blobs(centre, radius, float(sigma_max))


def node_coords(n_p: int, lo: float, hi: float) -> np.ndarray:
    """Vertex-aligned grid nodes spanning [lo, hi] (both faces included)."""
    return lo + np.arange(n_p, dtype=np.float64) * ((hi - lo) / (n_p - 1))


def bake_sigma_planes(n_p: int, blobs: Blobs, dtype=np.float32,
                      bmin=BOX_MIN, bmax=BOX_MAX,
                      s_frac: float = 0.25, rho_frac: float = 0.6) -> List[np.ndarray]:
    """Per-plane density factors: sum over blobs of
    sigma_max^(1/3) * exp(-(da^2 + db^2) / (4 s^2)), cut to 0 beyond rho."""
    amp = blobs.sigma_max ** (1.0 / 3.0)
    planes = []
    for (ra, rb) in PLANE_AXES:
        xa = node_coords(n_p, bmin[ra], bmax[ra])
        xb = node_coords(n_p, bmin[rb], bmax[rb])
        acc = np.zeros((n_p, n_p), dtype=np.float64)
        step_a = (bmax[ra] - bmin[ra]) / (n_p - 1)
        step_b = (bmax[rb] - bmin[rb]) / (n_p - 1)
        for c, r in zip(blobs.centre, blobs.radius):
            s = s_frac * r
            rho = rho_frac * r
            ca, cb = c[ra], c[rb]
            a0 = max(0, int(math.floor((ca - rho - bmin[ra]) / step_a)))
            a1 = min(n_p - 1, int(math.ceil((ca + rho - bmin[ra]) / step_a)))
            b0 = max(0, int(math.floor((cb - rho - bmin[rb]) / step_b)))
            b1 = min(n_p - 1, int(math.ceil((cb + rho - bmin[rb]) / step_b)))
            if a0 > a1 or b0 > b1:
                continue
            da = xa[a0:a1 + 1, None] - ca
            db = xb[None, b0:b1 + 1] - cb
            r2 = da * da + db * db
            f = amp * np.exp(-r2 / (4.0 * s * s))
            f[r2 > rho * rho] = 0.0
            acc[a0:a1 + 1, b0:b1 + 1] += f
        planes.append(acc.astype(dtype))
    return planes


def uniform_pm1(shape, dtype, rng: np.random.Generator, chunk_rows: int = 64) -> np.ndarray:
    """Values uniform in [-1, 1], rounded once from float32 to `dtype`,
    generated in row chunks so that large caches never hold float64 copies."""
    out = np.empty(shape, dtype=dtype)
    rows = shape[0]
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        v = rng.random(size=(r1 - r0,) + tuple(shape[1:]), dtype=np.float32)
        v *= 2.0
        v -= 1.0
        out[r0:r1] = v.astype(dtype)
    return out


def np_dtype(name: str):
    return {"f32": np.float32, "f16": np.float16}[name]


def bake_linear_sigma_planes(n_p: int, blobs: Blobs, channels: int, dtype=np.float32,
                             bmin=BOX_MIN, bmax=BOX_MAX, s_frac: float = 0.25,
                             rho_frac: float = 0.6) -> List[np.ndarray]:
    """Planar features for the linear decoder: blob b adds its planar
    Gaussian exp(-(da^2 + db^2) / (4 s^2)) (cut to 0 beyond rho) to channel
    b mod channels of every plane.  With all-ones weights and a threshold
    bias (linear_sigma_map) a point is dense only where its three planar
    projections all lie near blobs."""
    planes = []
    for (ra, rb) in PLANE_AXES:
        xa = node_coords(n_p, bmin[ra], bmax[ra])
        xb = node_coords(n_p, bmin[rb], bmax[rb])
        acc = np.zeros((n_p, n_p, channels), dtype=np.float64)
        step_a = (bmax[ra] - bmin[ra]) / (n_p - 1)
        step_b = (bmax[rb] - bmin[rb]) / (n_p - 1)
        for k, (c, r) in enumerate(zip(blobs.centre, blobs.radius)):
            s = s_frac * r
            rho = rho_frac * r
            ca, cb = c[ra], c[rb]
            a0 = max(0, int(math.floor((ca - rho - bmin[ra]) / step_a)))
            a1 = min(n_p - 1, int(math.ceil((ca + rho - bmin[ra]) / step_a)))
            b0 = max(0, int(math.floor((cb - rho - bmin[rb]) / step_b)))
            b1 = min(n_p - 1, int(math.ceil((cb + rho - bmin[rb]) / step_b)))
            if a0 > a1 or b0 > b1:
                continue
            da = xa[a0:a1 + 1, None] - ca
            db = xb[None, b0:b1 + 1] - cb
            r2 = da * da + db * db
            f = np.exp(-r2 / (4.0 * s * s))
            f[r2 > rho * rho] = 0.0
            acc[a0:a1 + 1, b0:b1 + 1, k % channels] += f
        planes.append(acc.astype(dtype))
    return planes


@dataclasses.dataclass
class LinearDecoder:
    """Eq. 5 parameters: sigma = W_sigma concat(sigma^xy, sigma^yz, sigma^zx)
    + b_sigma and, for each k in (u, v, w), k = W_k concat(k^xy, k^yz, k^zx)
    + b_k.  Shapes: w_sigma [3 Ds], b_sigma scalar, w_uvw [3][D][3D],
    b_uvw [3][D] (binary32)."""
    w_sigma: np.ndarray
    b_sigma: float
    w_uvw: np.ndarray
    b_uvw: np.ndarray


def linear_decoder(channels: int, D: int, sigma_max: float, seed: int,
                   threshold: float = 2.2) -> LinearDecoder:
    """Density weights scale * U(0.8, 1.2) per channel, with scale such that
    a point sitting on one blob in all three planes (feature sum 3) gets
    about sigma_max, and a bias that cuts everything below a feature sum of
    about `threshold`; radiance maps uniform in +-1/sqrt(3D), biases in
    +-0.1."""
    scale = sigma_max / (3.0 - threshold)
    rng = np.random.Generator(np.random.PCG64(seed))
    w_sigma = (scale * rng.uniform(0.8, 1.2, size=3 * channels)).astype(np.float32)
    b_sigma = float(np.float32(-scale * threshold))
    lim = 1.0 / math.sqrt(3 * D)
    w_uvw = rng.uniform(-lim, lim, size=(3, D, 3 * D)).astype(np.float32)
    b_uvw = rng.uniform(-0.1, 0.1, size=(3, D)).astype(np.float32)
    return LinearDecoder(w_sigma, b_sigma, w_uvw, b_uvw)


@dataclasses.dataclass
class Scene:
    """Everything one render call needs, as host arrays."""
    config: Config
    sigma: List[np.ndarray]
    uvw: List[np.ndarray]
    beta: np.ndarray
    poses: np.ndarray
    near: float = NEAR
    far: float = FAR
    bbox_min: tuple = BOX_MIN
    bbox_max: tuple = BOX_MAX
    seed: int = 0
    decoder: Optional[LinearDecoder] = None   # set for the linear (alt) decoder
    ndc_near: float = 0.0                     # > 0: rays marched in NDC

    @property
    def intrinsics(self):
        c = self.config
        return dict(fx=c.fx, fy=c.fx, cx=c.width / 2.0, cy=c.height / 2.0,
                    width=c.width, height=c.height)

    def cache_nbytes(self) -> int:
        """Bytes of the cache arrays (Sec. 3.3: 3 n_p^2 (3D + D_sigma) values
        plus n_d^2 D; the linear decoder's weights are not counted)."""
        return (sum(a.nbytes for a in self.sigma) + sum(a.nbytes for a in self.uvw)
                + self.beta.nbytes)


def make_scene(name_or_config, n_poses: Optional[int] = None) -> Scene:
    """Build the seeded inputs of one named workload ("tiny", "paper",
    "large", "batch", "stress") or of a Config."""
    cfg = CONFIGS[name_or_config] if isinstance(name_or_config, str) else name_or_config
    if n_poses is not None:
        cfg = dataclasses.replace(cfg, n_poses=n_poses)
    n = cfg.number
    dt = np_dtype(cfg.dtype)
    sdt = np_dtype(cfg.sigma_dtype or cfg.dtype)
    if cfg.forward:
        return _forward_scene(cfg)
    blobs = make_blobs(cfg.n_blobs, cfg.sigma_max, cfg.r_min, cfg.r_max, 1000 + n)
    decoder = None
    if cfg.sigma_channels > 0:
        sigma = bake_linear_sigma_planes(cfg.n_p, blobs, cfg.sigma_channels, sdt)
        decoder = linear_decoder(cfg.sigma_channels, cfg.D, cfg.sigma_max, 6000 + n)
    else:
        sigma = bake_sigma_planes(cfg.n_p, blobs, sdt)
    rng_uvw = np.random.Generator(np.random.PCG64(2000 + n))
    uvw = [uniform_pm1((cfg.n_p, cfg.n_p, 3 * cfg.D), dt, rng_uvw) for _ in range(3)]
    rng_beta = np.random.Generator(np.random.PCG64(3000 + n))
    beta = uniform_pm1((cfg.n_theta, cfg.n_phi, cfg.D), dt, rng_beta)
    poses = single_pose() if cfg.n_poses == 1 else spiral_poses(cfg.n_poses)
    return Scene(cfg, sigma, uvw, beta, poses, seed=4000 + n, decoder=decoder)


NDC_BOX = ((-1.0, -1.0, -1.0), (1.0, 1.0, 1.0))
NDC_NEAR = 1.0


def forward_pose(dx: float = 0.0, dy: float = 0.0, yaw_deg: float = 0.0, pitch_deg: float = 0.0):
    """Camera near the origin looking down -z (the frame of a forward-facing
    capture), moved by (dx, dy) and turned by small yaw / pitch angles."""
    cy, sy = math.cos(math.radians(yaw_deg)), math.sin(math.radians(yaw_deg))
    cp, sp = math.cos(math.radians(pitch_deg)), math.sin(math.radians(pitch_deg))
    Ry = np.array([[cy, 0, sy], [0, 1, 0], [-sy, 0, cy]])
    Rx = np.array([[1, 0, 0], [0, cp, -sp], [0, sp, cp]])
    P = np.zeros((3, 4))
    P[:, :3] = Ry @ Rx
    P[:, 3] = (dx, dy, 0.0)
    return P.astype(np.float32)


def forward_poses(n: int, seed: int = 5100) -> np.ndarray:
    """n forward-facing views: small seeded offsets (+-0.1) and turns (+-5 deg);
    the first is the reference view at the origin."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = [forward_pose()]
    for _ in range(n - 1):
        out.append(forward_pose(*rng.uniform(-0.1, 0.1, 2), *rng.uniform(-5.0, 5.0, 2)))
    return np.stack(out)


def _forward_scene(cfg: Config) -> Scene:
    """Forward-facing (LLFF-shaped) inputs: the caches span the NDC box
    [-1, 1]^3 of a camera looking down -z with near plane 1 (samples t' in
    [0, 1) from the near plane to infinity).  Blobs sit in NDC at x', y' in
    [-0.7, 0.7] and z' in [-0.6, 0.95] (world depths 1.25 to 40)."""
    n = cfg.number
    dt = np_dtype(cfg.dtype)
    sdt = np_dtype(cfg.sigma_dtype or cfg.dtype)
    rng = np.random.Generator(np.random.PCG64(1000 + n))
    centre = np.stack([rng.uniform(-0.7, 0.7, cfg.n_blobs), rng.uniform(-0.7, 0.7, cfg.n_blobs),
                       rng.uniform(-0.6, 0.95, cfg.n_blobs)], axis=1)
    blobs = Blobs(centre, rng.uniform(cfg.r_min, cfg.r_max, cfg.n_blobs), float(cfg.sigma_max))
    lo, hi = NDC_BOX
    sigma = bake_sigma_planes(cfg.n_p, blobs, sdt, bmin=lo, bmax=hi)
    rng_uvw = np.random.Generator(np.random.PCG64(2000 + n))
    uvw = [uniform_pm1((cfg.n_p, cfg.n_p, 3 * cfg.D), dt, rng_uvw) for _ in range(3)]
    rng_beta = np.random.Generator(np.random.PCG64(3000 + n))
    beta = uniform_pm1((cfg.n_theta, cfg.n_phi, cfg.D), dt, rng_beta)
    poses = forward_poses(cfg.n_poses)
    return Scene(cfg, sigma, uvw, beta, poses, near=0.0, far=1.0, bbox_min=lo, bbox_max=hi,
                 seed=4000 + n, ndc_near=NDC_NEAR)


# --------------------------------------------------------------------------
# cache generation: synthetic network weights (no trained weights exist here)

@dataclasses.dataclass(frozen=True)
class GenConfig:
    """One cache-generation workload: grid sizes and network shapes
    (Sec. 3.4: position networks of 6 layers x 256 units, direction network
    of 4 layers x 128 units; NeRF encodings with 10 and 4 frequencies)."""
    name: str
    number: int
    n_p: int
    n_theta: int
    n_phi: int
    D: int = 8
    pos_layers: int = 6
    pos_width: int = 256
    dir_layers: int = 4
    dir_width: int = 128
    pos_freq: int = 10
    dir_freq: int = 4

    @property
    def pos_in(self) -> int:
        return 2 * (1 + 2 * self.pos_freq)

    @property
    def dir_in(self) -> int:
        return 3 * (1 + 2 * self.dir_freq)

    @property
    def pos_out(self) -> int:
        return 2 + 6 * self.D


GEN_CONFIGS = {
    "gen_tiny": GenConfig("gen_tiny", 11, 32, 16, 16),
    # the paper's 512 cache (n_d = 64 on the synthetic scenes, Sec. 3.3)
    "gen_512": GenConfig("gen_512", 12, 512, 64, 64),
    # the 1K cache whose generation Table 4 times
    "gen_1k": GenConfig("gen_1k", 13, 1024, 64, 64),
}


def mlp_weights(sizes, seed: int, out_scale: float = 1.0):
    """[(W [out][in] binary16, b [out] binary32), ...] for the layer sizes
    sizes[0] -> sizes[1] -> ... : hidden layers He-uniform
    (+-sqrt(6 / fan_in)), the last layer uniform in +-out_scale/sqrt(fan_in);
    biases uniform in +-0.1."""
    rng = np.random.Generator(np.random.PCG64(seed))
    layers = []
    for n, (fi, fo) in enumerate(zip(sizes[:-1], sizes[1:])):
        last = n == len(sizes) - 2
        lim = out_scale / math.sqrt(fi) if last else math.sqrt(6.0 / fi)
        W = rng.uniform(-lim, lim, size=(fo, fi)).astype(np.float16)
        b = rng.uniform(-0.1, 0.1, size=fo).astype(np.float32)
        layers.append((W, b))
    return layers


@dataclasses.dataclass
class GenScene:
    config: GenConfig
    pos: list          # three layer lists, planes xy, yz, zx
    dir: list
    bbox_min: tuple = BOX_MIN
    bbox_max: tuple = BOX_MAX


def make_gen_scene(name_or_config) -> GenScene:
    cfg = GEN_CONFIGS[name_or_config] if isinstance(name_or_config, str) else name_or_config
    n = cfg.number
    pos_sizes = [cfg.pos_in] + [cfg.pos_width] * cfg.pos_layers + [cfg.pos_out]
    dir_sizes = [cfg.dir_in] + [cfg.dir_width] * cfg.dir_layers + [cfg.D]
    pos = [mlp_weights(pos_sizes, 7000 + 10 * n + j, out_scale=1.5) for j in range(3)]
    dirw = mlp_weights(dir_sizes, 7000 + 10 * n + 5, out_scale=1.5)
    return GenScene(cfg, pos, dirw)

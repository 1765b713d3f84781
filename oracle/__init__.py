"""CPU oracle for the cached SqueezeNeRF renderer -- TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its binding)
never does.  The arithmetic lives in ``oracle.c`` (plain C, binary32 exact
path without fused multiply-add, binary64 value path); this module only
compiles it and marshals numpy arrays.

Functions and the passages they follow:
  render        -- Eq. 1 compositing of Eq. 4 (or Eq. 5) / Eq. 2 cached
                   fields along pinhole rays (Sec. 3.1, 3.2, 3.3, 3.4)
  tau_eps_q     -- transmittance threshold T >= eps as a fixed-point optical
                   depth bound
  half_to_double, splitmix64 -- input decoding and the stratified-sampling
                   counter generator (Steele, Lea & Flood 2014)
  cache_nbytes  -- storage formula of Sec. 3.3
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SOURCES = [os.path.join(_HERE, "oracle.c")]

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
          "-shared", "-pthread", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    """Compile liboracle.so with gcc (always recompiles)."""
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, *SOURCES, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    global _lib
    _lib = None
    return LIB_PATH


class _Scene(ctypes.Structure):
    _fields_ = [("n_p", ctypes.c_int32), ("D", ctypes.c_int32),
                ("n_theta", ctypes.c_int32), ("n_phi", ctypes.c_int32),
                ("sigma_f16", ctypes.c_int32), ("uvw_f16", ctypes.c_int32),
                ("beta_f16", ctypes.c_int32), ("stratified", ctypes.c_int32),
                ("bmin", ctypes.c_float * 3), ("bmax", ctypes.c_float * 3),
                ("t_eps", ctypes.c_float), ("pad0", ctypes.c_int32),
                ("seed", ctypes.c_uint64),
                ("sigma", ctypes.c_void_p * 3), ("uvw", ctypes.c_void_p * 3),
                ("beta", ctypes.c_void_p),
                ("d_sigma", ctypes.c_int32), ("b_sigma", ctypes.c_float),
                ("w_sigma", ctypes.c_void_p), ("w_uvw", ctypes.c_void_p),
                ("b_uvw", ctypes.c_void_p)]


class _Camera(ctypes.Structure):
    _fields_ = [("fx", ctypes.c_float), ("fy", ctypes.c_float),
                ("cx", ctypes.c_float), ("cy", ctypes.c_float),
                ("width", ctypes.c_int32), ("height", ctypes.c_int32),
                ("ndc_near", ctypes.c_float), ("pad", ctypes.c_int32)]


RAY_DTYPE = np.dtype([("rgb", np.float64, (3,)), ("depth", np.float64),
                      ("acc", np.float64), ("tau_end", np.int64),
                      ("stop", np.uint32), ("n_inbox", np.uint32),
                      ("n_occ", np.uint32), ("hash", np.uint32)])
assert RAY_DTYPE.itemsize == 64

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        lib = ctypes.CDLL(LIB_PATH)
        lib.oracle_render.restype = ctypes.c_int
        lib.oracle_render.argtypes = [ctypes.POINTER(_Scene), ctypes.c_void_p, ctypes.c_int32,
                                      ctypes.POINTER(_Camera), ctypes.c_float, ctypes.c_float,
                                      ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_void_p, ctypes.c_int32]
        lib.oracle_tau_eps_q.restype = ctypes.c_int64
        lib.oracle_tau_eps_q.argtypes = [ctypes.c_float]
        lib.oracle_half_to_double.restype = ctypes.c_double
        lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_splitmix64.restype = ctypes.c_uint64
        lib.oracle_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        _lib = lib
    return _lib


def tau_eps_q(eps: float) -> int:
    return int(_load().oracle_tau_eps_q(float(eps)))


def half_to_double(bits: int) -> float:
    return float(_load().oracle_half_to_double(int(bits)))


def splitmix64(seed: int, counter: int) -> int:
    return int(_load().oracle_splitmix64(int(seed), int(counter)))


def cache_nbytes(n_p: int, D: int, n_theta: int, n_phi: int,
                 sigma_bytes: int, uvw_bytes: int, beta_bytes: int, d_sigma: int = 1) -> int:
    """Sec. 3.3: three n_p x n_p planes of sigma^j (1 value; D_sigma values
    for the Eq. 5 decoder) and u^j, v^j, w^j (D values each), plus
    n_theta x n_phi x D direction weights."""
    return (3 * n_p * n_p * (d_sigma * sigma_bytes + 3 * D * uvw_bytes)
            + n_theta * n_phi * D * beta_bytes)


def _dtype_flag(a: np.ndarray) -> int:
    if a.dtype == np.float16:
        return 1
    if a.dtype == np.float32:
        return 0
    raise TypeError(f"cache arrays must be float16 or float32, got {a.dtype}")


def render(sigma: Sequence[np.ndarray], uvw: Sequence[np.ndarray], beta: np.ndarray,
           poses: np.ndarray, intrinsics: dict, near: float, far: float, n_samples: int,
           bbox_min, bbox_max, t_eps: float = 1e-4, stratified: bool = False,
           seed: int = 0, ray_ids: Optional[np.ndarray] = None,
           n_threads: Optional[int] = None, decoder=None, ndc_near: float = 0.0) -> np.ndarray:
    """Render rays on the CPU; returns a structured array of RAY_DTYPE
    (rgb, depth, acc, tau_end, stop, n_inbox, n_occ, hash), one per ray,
    in ray-id order ((b*H + v)*W + u) or in the order of `ray_ids`.

    decoder: None for Eq. 4, or an object with w_sigma [3 D_sigma],
    b_sigma, w_uvw [3][D][3D] and b_uvw [3][D] for Eq. 5; then each
    sigma[j] is [n_p][n_p][D_sigma].  ndc_near > 0 marches in normalized
    device coordinates with that near plane (forward-facing captures);
    near/far are then the NDC ray parameters, usually 0 and 1."""
    lib = _load()
    sigma = [np.ascontiguousarray(a) for a in sigma]
    uvw = [np.ascontiguousarray(a) for a in uvw]
    beta = np.ascontiguousarray(beta)
    poses = np.ascontiguousarray(poses, dtype=np.float32).reshape(-1, 3, 4)
    n_p = sigma[0].shape[0]
    D = uvw[0].shape[-1] // 3
    d_sigma = 0 if decoder is None else sigma[0].shape[2]
    want = (n_p, n_p) if decoder is None else (n_p, n_p, d_sigma)
    for a in sigma:
        assert a.shape == want and a.dtype == sigma[0].dtype
    for a in uvw:
        assert a.shape == (n_p, n_p, 3 * D) and a.dtype == uvw[0].dtype
    assert beta.ndim == 3 and beta.shape[2] == D

    sc = _Scene()
    sc.n_p, sc.D = n_p, D
    sc.n_theta, sc.n_phi = beta.shape[0], beta.shape[1]
    sc.sigma_f16, sc.uvw_f16, sc.beta_f16 = _dtype_flag(sigma[0]), _dtype_flag(uvw[0]), _dtype_flag(beta)
    sc.stratified = 1 if stratified else 0
    for r in range(3):
        sc.bmin[r] = bbox_min[r]
        sc.bmax[r] = bbox_max[r]
    sc.t_eps = t_eps
    sc.seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    for j in range(3):
        sc.sigma[j] = sigma[j].ctypes.data
        sc.uvw[j] = uvw[j].ctypes.data
    sc.beta = beta.ctypes.data
    if decoder is not None:
        w_sigma = np.ascontiguousarray(decoder.w_sigma, dtype=np.float32)
        w_uvw = np.ascontiguousarray(decoder.w_uvw, dtype=np.float32)
        b_uvw = np.ascontiguousarray(decoder.b_uvw, dtype=np.float32)
        assert d_sigma >= 1 and w_sigma.shape == (3 * d_sigma,)
        assert w_uvw.shape == (3, D, 3 * D) and b_uvw.shape == (3, D)
        sc.d_sigma = d_sigma
        sc.b_sigma = float(decoder.b_sigma)
        sc.w_sigma = w_sigma.ctypes.data
        sc.w_uvw = w_uvw.ctypes.data
        sc.b_uvw = b_uvw.ctypes.data

    cam = _Camera(float(intrinsics["fx"]), float(intrinsics["fy"]), float(intrinsics["cx"]),
                  float(intrinsics["cy"]), int(intrinsics["width"]), int(intrinsics["height"]),
                  float(ndc_near), 0)
    total = poses.shape[0] * cam.width * cam.height
    if ray_ids is None:
        ids_ptr, n = None, total
    else:
        ray_ids = np.ascontiguousarray(ray_ids, dtype=np.int64)
        ids_ptr, n = ray_ids.ctypes.data, ray_ids.size
    out = np.zeros(n, dtype=RAY_DTYPE)
    if n_threads is None:
        n_threads = os.cpu_count() or 1
    rc = lib.oracle_render(ctypes.byref(sc), poses.ctypes.data, poses.shape[0], ctypes.byref(cam),
                           float(near), float(far), int(n_samples), ids_ptr, n,
                           out.ctypes.data if n else None, int(n_threads))
    if rc != 0:
        raise ValueError("oracle_render rejected its arguments")
    return out


def render_scene(scene, ray_ids=None, n_threads=None, n_samples=None, t_eps=None,
                 stratified=None, poses=None) -> np.ndarray:
    """render() with the arguments taken from a scene object's attributes
    (sigma, uvw, beta, poses, intrinsics, near, far, bbox_min, bbox_max,
    config.n_samples / t_eps / stratified, seed)."""
    cfg = scene.config
    return render(scene.sigma, scene.uvw, scene.beta,
                  scene.poses if poses is None else poses, scene.intrinsics,
                  scene.near, scene.far, cfg.n_samples if n_samples is None else n_samples,
                  scene.bbox_min, scene.bbox_max,
                  t_eps=cfg.t_eps if t_eps is None else t_eps,
                  stratified=cfg.stratified if stratified is None else stratified,
                  seed=scene.seed, ray_ids=ray_ids, n_threads=n_threads,
                  decoder=getattr(scene, "decoder", None),
                  ndc_near=getattr(scene, "ndc_near", 0.0))

"""ctypes binding of libsqn.so (include/sqn.h) over torch device tensors.

Argument marshalling only: every step of the render runs in the HIP
library.  torch provides device memory and the current stream.  Importing
this module loads libsqn.so and raises if it has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsqn.so")

SQN_OK, SQN_ERR_INVALID_ARG, SQN_ERR_OUT_OF_MEMORY, SQN_ERR_DEVICE, SQN_ERR_UNSUPPORTED = range(5)
SQN_F32, SQN_F16 = 0, 1

EXPORTS = ("sqn_create_caches", "sqn_create_linear_caches", "sqn_recreate_caches", "sqn_render", "sqn_render_stats",
           "sqn_set_lanes_per_ray", "sqn_tune_lanes_per_ray", "sqn_set_centre_block",
           "sqn_set_empty_space_skipping", "sqn_set_ndc", "sqn_cache_device_bytes",
           "sqn_destroy", "sqn_status_string", "sqn_last_error", "sqn_create_networks",
           "sqn_generate_caches", "sqn_networks_device_bytes", "sqn_destroy_networks")


class CacheDesc(ctypes.Structure):
    _fields_ = [("n_p", ctypes.c_int32), ("D", ctypes.c_int32),
                ("n_theta", ctypes.c_int32), ("n_phi", ctypes.c_int32),
                ("sigma_dtype", ctypes.c_int32), ("uvw_dtype", ctypes.c_int32),
                ("beta_dtype", ctypes.c_int32), ("stratified", ctypes.c_int32),
                ("bbox_min", ctypes.c_float * 3), ("bbox_max", ctypes.c_float * 3),
                ("t_eps", ctypes.c_float), ("reserved", ctypes.c_int32),
                ("seed", ctypes.c_uint64)]


class LinearDecoder(ctypes.Structure):
    _fields_ = [("d_sigma", ctypes.c_int32), ("b_sigma", ctypes.c_float),
                ("w_sigma", ctypes.c_void_p), ("w_uvw", ctypes.c_void_p),
                ("b_uvw", ctypes.c_void_p)]


class MLPDesc(ctypes.Structure):
    _fields_ = [("n_hidden", ctypes.c_int32), ("width", ctypes.c_int32),
                ("n_in", ctypes.c_int32), ("n_out", ctypes.c_int32),
                ("weights", ctypes.POINTER(ctypes.c_void_p)),
                ("biases", ctypes.POINTER(ctypes.c_void_p))]


class Intrinsics(ctypes.Structure):
    _fields_ = [("fx", ctypes.c_float), ("fy", ctypes.c_float),
                ("cx", ctypes.c_float), ("cy", ctypes.c_float),
                ("width", ctypes.c_int32), ("height", ctypes.c_int32)]


class SqnError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{status_string(status)}: {detail}")
        self.status = status
        self.detail = detail


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first "
                          "(python -m paper_2204_02585_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    lib.sqn_create_caches.restype = ctypes.c_int
    lib.sqn_create_caches.argtypes = [ctypes.POINTER(CacheDesc), ctypes.POINTER(vp),
                                      ctypes.POINTER(vp), vp, vp, ctypes.POINTER(vp)]
    lib.sqn_create_linear_caches.restype = ctypes.c_int
    lib.sqn_create_linear_caches.argtypes = [ctypes.POINTER(CacheDesc), ctypes.POINTER(LinearDecoder),
                                             ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp,
                                             ctypes.POINTER(vp)]
    lib.sqn_recreate_caches.restype = ctypes.c_int
    lib.sqn_recreate_caches.argtypes = [vp, ctypes.POINTER(CacheDesc), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                        vp, vp]
    lib.sqn_create_networks.restype = ctypes.c_int
    lib.sqn_create_networks.argtypes = [ctypes.POINTER(MLPDesc), ctypes.POINTER(MLPDesc), i32, i32, i32,
                                        vp, ctypes.POINTER(vp)]
    lib.sqn_generate_caches.restype = ctypes.c_int
    lib.sqn_generate_caches.argtypes = [vp, ctypes.POINTER(CacheDesc), ctypes.POINTER(vp),
                                        ctypes.POINTER(vp), vp, vp]
    lib.sqn_networks_device_bytes.restype = ctypes.c_size_t
    lib.sqn_networks_device_bytes.argtypes = [vp]
    lib.sqn_destroy_networks.restype = None
    lib.sqn_destroy_networks.argtypes = [vp]
    lib.sqn_render.restype = ctypes.c_int
    lib.sqn_render.argtypes = [vp, vp, i32, ctypes.POINTER(Intrinsics), f32, f32, i32, vp, vp, vp]
    lib.sqn_render_stats.restype = ctypes.c_int
    lib.sqn_render_stats.argtypes = [vp, vp, i32, ctypes.POINTER(Intrinsics), f32, f32, i32,
                                     vp, vp, vp, vp]
    lib.sqn_set_lanes_per_ray.restype = ctypes.c_int
    lib.sqn_set_lanes_per_ray.argtypes = [vp, i32]
    lib.sqn_set_centre_block.restype = ctypes.c_int
    lib.sqn_set_centre_block.argtypes = [vp, f32]
    lib.sqn_tune_lanes_per_ray.restype = ctypes.c_int
    lib.sqn_tune_lanes_per_ray.argtypes = [vp, vp, i32, ctypes.POINTER(Intrinsics), f32, f32, i32, vp, vp, vp,
                                           ctypes.POINTER(i32), ctypes.POINTER(f32)]
    lib.sqn_set_empty_space_skipping.restype = ctypes.c_int
    lib.sqn_set_empty_space_skipping.argtypes = [vp, i32]
    lib.sqn_set_ndc.restype = ctypes.c_int
    lib.sqn_set_ndc.argtypes = [vp, f32]
    lib.sqn_cache_device_bytes.restype = ctypes.c_size_t
    lib.sqn_cache_device_bytes.argtypes = [vp]
    lib.sqn_destroy.restype = None
    lib.sqn_destroy.argtypes = [vp]
    lib.sqn_status_string.restype = ctypes.c_char_p
    lib.sqn_status_string.argtypes = [ctypes.c_int]
    lib.sqn_last_error.restype = ctypes.c_char_p
    lib.sqn_last_error.argtypes = []
    return lib


lib = _load()


def status_string(status: int) -> str:
    return lib.sqn_status_string(int(status)).decode()


def last_error() -> str:
    return lib.sqn_last_error().decode()


def _check(status: int) -> None:
    if status != SQN_OK:
        raise SqnError(status, last_error())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float16:
        return SQN_F16
    if t.dtype == torch.float32:
        return SQN_F32
    raise TypeError(f"cache tensors must be float16 or float32, got {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _poses_arg(poses: torch.Tensor) -> torch.Tensor:
    """float32 [B,3,4] camera-to-world on a CUDA device, contiguous; [B,4,4]
    poses lose their last row."""
    if poses.dtype != torch.float32:
        raise TypeError(f"poses must be float32, got {poses.dtype}")
    if poses.device.type != "cuda":
        raise ValueError("poses must live on a CUDA device")
    if poses.dim() != 3 or poses.shape[1:] not in ((3, 4), (4, 4)):
        raise ValueError(f"poses must have shape [B,3,4] (or [B,4,4]), got {tuple(poses.shape)}")
    return poses[:, :3, :].contiguous()


def _output_arg(t: torch.Tensor, shape, device, name: str) -> None:
    if t.dtype != torch.float32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or t.device != device:
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {tuple(shape)} on {device}")


def _intrinsics(intr: dict) -> Intrinsics:
    return Intrinsics(float(intr["fx"]), float(intr["fy"]), float(intr["cx"]), float(intr["cy"]),
                      int(intr["width"]), int(intr["height"]))


def _cache_args(sigma, uvw, beta, bbox_min, bbox_max, t_eps, stratified, seed, stream):
    """sqn_cache_desc and plane pointer arrays for cache tensors on one
    device.  Copies made to make a tensor contiguous are ordered before the
    library's work on `stream`."""
    sigma = [s.contiguous() for s in sigma]
    uvw = [u.contiguous() for u in uvw]
    beta = beta.contiguous()
    dev = beta.device
    if len(sigma) != 3 or len(uvw) != 3:
        raise ValueError("three sigma planes and three uvw planes are needed (xy, yz, zx)")
    for t in (*sigma, *uvw, beta):
        if t.device != dev or dev.type != "cuda":
            raise ValueError("cache tensors must all live on one CUDA device")
    n_p, D = sigma[0].shape[0], uvw[0].shape[-1] // 3
    if (any(t.shape[:2] != (n_p, n_p) or t.dtype != sigma[0].dtype or t.dim() != sigma[0].dim() for t in sigma)
            or any(t.shape != (n_p, n_p, 3 * D) or t.dtype != uvw[0].dtype for t in uvw)
            or uvw[0].shape[-1] % 3 != 0 or beta.dim() != 3 or beta.shape[2] != D):
        raise ValueError("cache shapes: sigma [n_p, n_p] (or [n_p, n_p, D_sigma]), uvw [n_p, n_p, 3D], "
                         "beta [n_theta, n_phi, D], one dtype per kind")
    _order_after_current(stream, *sigma, *uvw, beta)
    desc = CacheDesc()
    desc.n_p, desc.D = sigma[0].shape[0], uvw[0].shape[-1] // 3
    desc.n_theta, desc.n_phi = beta.shape[0], beta.shape[1]
    desc.sigma_dtype, desc.uvw_dtype, desc.beta_dtype = (_dtype_code(sigma[0]), _dtype_code(uvw[0]),
                                                         _dtype_code(beta))
    desc.stratified = 1 if stratified else 0
    for r in range(3):
        desc.bbox_min[r] = bbox_min[r]
        desc.bbox_max[r] = bbox_max[r]
    desc.t_eps = t_eps
    desc.reserved = 0
    desc.seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    sp = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in sigma])
    up = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in uvw])
    return desc, sigma, uvw, beta, sp, up


def _order_after_current(stream, *tensors) -> None:
    """Make `stream` wait for the work already queued on torch's current
    stream (the copies .contiguous() or .to() may just have queued there),
    and tell torch's allocator that `tensors` are in use on `stream`."""
    if stream is not None and stream != torch.cuda.current_stream():
        stream.wait_stream(torch.cuda.current_stream())
        for t in tensors:
            if t is not None:
                t.record_stream(stream)


class Caches:
    """Library-owned device copy of the SqueezeNeRF caches (sqn_create_caches,
    or sqn_create_linear_caches when `decoder` is given: an object with
    w_sigma [3 D_sigma], b_sigma, w_uvw [3][D][3D] and b_uvw [3][D], and
    sigma planes of shape [n_p][n_p][D_sigma])."""

    def __init__(self, sigma: Sequence[torch.Tensor], uvw: Sequence[torch.Tensor],
                 beta: torch.Tensor, bbox_min, bbox_max, t_eps: float = 1e-4,
                 stratified: bool = False, seed: int = 0, stream=None, decoder=None):
        self._h = ctypes.c_void_p(None)
        desc, sigma, uvw, beta, sp, up = _cache_args(sigma, uvw, beta, bbox_min, bbox_max, t_eps,
                                                     stratified, seed, stream)
        self.desc = desc
        D = desc.D
        if decoder is None:
            _check(lib.sqn_create_caches(ctypes.byref(desc), sp, up, _ptr(beta), _stream(stream),
                                         ctypes.byref(self._h)))
            return
        import numpy as np
        w_sigma = np.ascontiguousarray(decoder.w_sigma, dtype=np.float32)
        w_uvw = np.ascontiguousarray(decoder.w_uvw, dtype=np.float32)
        b_uvw = np.ascontiguousarray(decoder.b_uvw, dtype=np.float32)
        d_sigma = int(sigma[0].shape[2]) if sigma[0].dim() == 3 else 0
        # the library reads these host arrays at these sizes
        if (w_sigma.shape != (3 * d_sigma,) or w_uvw.shape != (3, D, 3 * D)
                or b_uvw.shape != (3, D)):
            raise ValueError("decoder weights do not match d_sigma and D")
        dec = LinearDecoder(d_sigma,
                            float(decoder.b_sigma), w_sigma.ctypes.data, w_uvw.ctypes.data,
                            b_uvw.ctypes.data)
        _check(lib.sqn_create_linear_caches(ctypes.byref(desc), ctypes.byref(dec), sp, up,
                                            _ptr(beta), _stream(stream), ctypes.byref(self._h)))

    @property
    def handle(self) -> ctypes.c_void_p:
        if not self._h:
            raise ValueError("caches have been destroyed")
        return self._h

    def recreate(self, sigma: Sequence[torch.Tensor], uvw: Sequence[torch.Tensor], beta: torch.Tensor,
                 bbox_min, bbox_max, t_eps: float = 1e-4, stratified: bool = False, seed: int = 0,
                 stream=None) -> None:
        """sqn_recreate_caches: new Eq. 4 caches in this handle's device
        memory, without allocating; the tensors must stay alive until
        `stream` has finished the call's work."""
        desc, sigma, uvw, beta, sp, up = _cache_args(sigma, uvw, beta, bbox_min, bbox_max, t_eps,
                                                     stratified, seed, stream)
        _check(lib.sqn_recreate_caches(self.handle, ctypes.byref(desc), sp, up, _ptr(beta), _stream(stream)))
        self.desc = desc

    @property
    def device_bytes(self) -> int:
        return int(lib.sqn_cache_device_bytes(self.handle))

    def set_lanes_per_ray(self, lanes: int) -> None:
        """1, 4 or 8 lanes of a wavefront per ray, or 0 to choose per call."""
        _check(lib.sqn_set_lanes_per_ray(self.handle, int(lanes)))

    def set_centre_block(self, fraction: float) -> None:
        """Hybrid launch of single views: the centred `fraction` of the image
        (per axis, in 16-pixel blocks) with four lanes per ray, the rest with
        one; 0 turns it off."""
        _check(lib.sqn_set_centre_block(self.handle, float(fraction)))

    def tune_lanes_per_ray(self, poses: torch.Tensor, intrinsics: dict, near: float, far: float,
                           n_samples: int, rgb_out: Optional[torch.Tensor] = None,
                           depth_out: Optional[torch.Tensor] = None, stream=None) -> int:
        """sqn_tune_lanes_per_ray: time the launch shapes on this batch, keep
        the fastest for later renders and return it: lanes per ray, or -1 for
        a hybrid launch, whose centre fraction is then in self.centre_block.
        Blocks; rgb_out / depth_out (allocated if not given) receive a
        render."""
        poses = _poses_arg(poses)
        B = poses.shape[0]
        H, W = int(intrinsics["height"]), int(intrinsics["width"])
        if rgb_out is None:
            rgb_out = torch.empty((B, H, W, 3), dtype=torch.float32, device=poses.device)
        if depth_out is None:
            depth_out = torch.empty((B, H, W), dtype=torch.float32, device=poses.device)
        _output_arg(rgb_out, (B, H, W, 3), poses.device, "rgb_out")
        _output_arg(depth_out, (B, H, W), poses.device, "depth_out")
        _order_after_current(stream, poses, rgb_out, depth_out)
        intr = _intrinsics(intrinsics)
        chosen, centre = ctypes.c_int32(0), ctypes.c_float(0.0)
        _check(lib.sqn_tune_lanes_per_ray(self.handle, _ptr(poses), B, ctypes.byref(intr), float(near),
                                          float(far), int(n_samples), _ptr(rgb_out), _ptr(depth_out),
                                          _stream(stream), ctypes.byref(chosen), ctypes.byref(centre)))
        self.centre_block = float(centre.value)
        return int(chosen.value)

    def set_empty_space_skipping(self, enable: bool) -> None:
        """Leaps over empty space (default) or a dense march."""
        _check(lib.sqn_set_empty_space_skipping(self.handle, 1 if enable else 0))

    def set_ndc(self, ndc_near: float) -> None:
        """Forward-facing rays in normalized device coordinates with near
        plane ndc_near (> 0), or world rays (0)."""
        _check(lib.sqn_set_ndc(self.handle, float(ndc_near)))

    def close(self) -> None:
        if self._h:
            lib.sqn_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def render(self, poses: torch.Tensor, intrinsics: dict, near: float, far: float,
               n_samples: int, rgb_out: Optional[torch.Tensor] = None,
               depth_out: Optional[torch.Tensor] = None, with_depth: bool = True, stream=None):
        """sqn_render; returns (rgb [B,H,W,3], depth [B,H,W] or None).
        poses: float32 [B,3,4] camera-to-world (or [B,4,4], whose last row is
        dropped) on the caches' device."""
        poses = _poses_arg(poses)
        B = poses.shape[0]
        H, W = int(intrinsics["height"]), int(intrinsics["width"])
        if rgb_out is None:
            rgb_out = torch.empty((B, H, W, 3), dtype=torch.float32, device=poses.device)
        if depth_out is None and with_depth:
            depth_out = torch.empty((B, H, W), dtype=torch.float32, device=poses.device)
        _output_arg(rgb_out, (B, H, W, 3), poses.device, "rgb_out")
        if depth_out is not None:
            _output_arg(depth_out, (B, H, W), poses.device, "depth_out")
        _order_after_current(stream, poses, rgb_out, depth_out)
        intr = _intrinsics(intrinsics)
        _check(lib.sqn_render(self.handle, _ptr(poses), B, ctypes.byref(intr), float(near),
                              float(far), int(n_samples), _ptr(rgb_out), _ptr(depth_out),
                              _stream(stream)))
        return rgb_out, depth_out

    def render_stats(self, poses: torch.Tensor, intrinsics: dict, near: float, far: float,
                     n_samples: int, stream=None):
        """sqn_render_stats; returns (rgb, depth, stats [B,H,W,4] int32 view of
        {stop, n_inbox, n_occ, hash}).  poses as for render()."""
        poses = _poses_arg(poses)
        B = poses.shape[0]
        H, W = int(intrinsics["height"]), int(intrinsics["width"])
        rgb = torch.empty((B, H, W, 3), dtype=torch.float32, device=poses.device)
        depth = torch.empty((B, H, W), dtype=torch.float32, device=poses.device)
        stats = torch.empty((B, H, W, 4), dtype=torch.int32, device=poses.device)
        _order_after_current(stream, poses, rgb, depth, stats)
        intr = _intrinsics(intrinsics)
        _check(lib.sqn_render_stats(self.handle, _ptr(poses), B, ctypes.byref(intr), float(near),
                                    float(far), int(n_samples), _ptr(rgb), _ptr(depth),
                                    _ptr(stats), _stream(stream)))
        return rgb, depth, stats


def caches_from_scene(scene, device="cuda", t_eps=None, stratified=None, stream=None) -> Caches:
    """Upload a scene's host arrays (see scenes.Scene) and create the caches."""
    cfg = scene.config
    sig = [torch.from_numpy(a).to(device) for a in scene.sigma]
    uvw = [torch.from_numpy(a).to(device) for a in scene.uvw]
    beta = torch.from_numpy(scene.beta).to(device)
    caches = Caches(sig, uvw, beta, scene.bbox_min, scene.bbox_max,
                    t_eps=cfg.t_eps if t_eps is None else t_eps,
                    stratified=cfg.stratified if stratified is None else stratified,
                    seed=scene.seed, stream=stream, decoder=getattr(scene, "decoder", None))
    if getattr(scene, "ndc_near", 0.0) > 0.0:
        caches.set_ndc(scene.ndc_near)
    return caches


# ---------------------------------------------------------------- cache generation

class _MLP:
    """Keeps the host arrays of one network alive while its descriptor is in
    use; the descriptor states the shapes the arrays really have."""

    def __init__(self, layers):
        import numpy as np
        self.W = [np.ascontiguousarray(W, dtype=np.float16) for W, _ in layers]
        self.b = [np.ascontiguousarray(b, dtype=np.float32) for _, b in layers]
        width = self.W[0].shape[0]
        for n, (W, b) in enumerate(zip(self.W, self.b)):
            fi = self.W[0].shape[1] if n == 0 else width
            fo = self.W[-1].shape[0] if n == len(self.W) - 1 else width
            if W.shape != (fo, fi) or b.shape != (fo,):
                raise ValueError(f"layer {n}: weight {W.shape} / bias {b.shape} do not chain")
        self.wp = (ctypes.c_void_p * len(self.W))(*[w.ctypes.data for w in self.W])
        self.bp = (ctypes.c_void_p * len(self.b))(*[b.ctypes.data for b in self.b])
        self.desc = MLPDesc(len(layers) - 1, width, self.W[0].shape[1], self.W[-1].shape[0],
                            ctypes.cast(self.wp, ctypes.POINTER(ctypes.c_void_p)),
                            ctypes.cast(self.bp, ctypes.POINTER(ctypes.c_void_p)))


class Networks:
    """Library-owned device copy of the position and direction networks
    (sqn_create_networks); layers are lists of (W [out][in] binary16,
    b [out] binary32)."""

    def __init__(self, pos_layers, dir_layers, D: int, pos_freq: int = 10, dir_freq: int = 4,
                 stream=None):
        self._h = ctypes.c_void_p(None)
        pos = [_MLP(l) for l in pos_layers]
        dirn = _MLP(dir_layers)
        arr = (MLPDesc * 3)(*[m.desc for m in pos])
        _check(lib.sqn_create_networks(arr, ctypes.byref(dirn.desc), int(D), int(pos_freq), int(dir_freq),
                                       _stream(stream), ctypes.byref(self._h)))
        self.D = D

    @property
    def handle(self) -> ctypes.c_void_p:
        if not self._h:
            raise ValueError("networks have been destroyed")
        return self._h

    @property
    def device_bytes(self) -> int:
        return int(lib.sqn_networks_device_bytes(self.handle))

    def generate(self, n_p: int, n_theta: int, n_phi: int, bbox_min, bbox_max,
                 sigma_dtype=torch.float32, uvw_dtype=torch.float16, beta_dtype=torch.float16,
                 out=None, stream=None, device="cuda"):
        """sqn_generate_caches; returns ([sigma^j], [uvw^j], beta) device tensors
        (or fills `out`, a tuple of that form)."""
        D = self.D
        if out is None:
            sig = [torch.empty((n_p, n_p), dtype=sigma_dtype, device=device) for _ in range(3)]
            uvw = [torch.empty((n_p, n_p, 3 * D), dtype=uvw_dtype, device=device) for _ in range(3)]
            beta = torch.empty((n_theta, n_phi, D), dtype=beta_dtype, device=device)
        else:
            sig, uvw, beta = out
        desc = CacheDesc()
        desc.n_p, desc.D, desc.n_theta, desc.n_phi = n_p, D, n_theta, n_phi
        desc.sigma_dtype, desc.uvw_dtype, desc.beta_dtype = (_dtype_code(sig[0]), _dtype_code(uvw[0]),
                                                             _dtype_code(beta))
        for r in range(3):
            desc.bbox_min[r] = bbox_min[r]
            desc.bbox_max[r] = bbox_max[r]
        desc.t_eps = 0.0
        sp = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in sig])
        up = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in uvw])
        _check(lib.sqn_generate_caches(self.handle, ctypes.byref(desc), sp, up, _ptr(beta), _stream(stream)))
        return sig, uvw, beta

    def close(self) -> None:
        if self._h:
            lib.sqn_destroy_networks(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def networks_from_gen_scene(gscene, stream=None) -> Networks:
    c = gscene.config
    return Networks(gscene.pos, gscene.dir, c.D, c.pos_freq, c.dir_freq, stream=stream)

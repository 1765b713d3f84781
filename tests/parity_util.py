"""Helpers shared by the GPU parity tests (imports torch and the binding
lazily so that CPU-only collection never loads the GPU library)."""
import numpy as np

# value tolerances: binary32 caches 1e-5 absolute, binary16 caches 1e-3
# absolute (the oracle reads the same binary16 values)
ATOL = {"f32": 1e-5, "f16": 1e-3}
# regression bound asserted beside them: the oracle reads the very binary16
# values the kernel reads, so both sides evaluate the same real numbers and
# only the kernel's binary32 value path (binary64 sums) separates them,
# bounded near 1e-6 whatever the cache dtype; 1e-5 flags a value-path
# regression that the 1e-3 criterion of binary16 caches would let through
REGRESSION_ATOL = 1e-5


def scene_atol(scene):
    return ATOL[scene.config.dtype]


# launch variants: library default (leaps, lanes chosen per call), leaps with
# 1, 4 or 8 lanes per ray, the hybrid launch (leaps; single views of the
# product decoder: the centred half of the image with four lanes per ray, the
# rest with one; other renders as "auto"), and the dense march with 1, 4 or 8
# lanes per ray
MODES = {"auto": (0, True), "skip1": (1, True), "skip4": (4, True), "skip8": (8, True), "hyb": (0, True, 0.5),
         "L1": (1, False), "L4": (4, False), "L8": (8, False)}


def gpu_render(scene, t_eps=None, poses=None, n_samples=None, stats=True, mode="auto", shape=None):
    """Render a scene through the C ABI in one of MODES, or in an explicit
    launch shape (lanes per ray, hybrid centre fraction) with leaps; returns
    numpy (rgb, depth, stats)."""
    import torch
    from paper_2204_02585_amd import binding
    caches = binding.caches_from_scene(scene, t_eps=t_eps)
    lanes, skip = MODES[mode][:2]
    centre = MODES[mode][2] if len(MODES[mode]) > 2 else 0.0
    if shape is not None:
        (lanes, centre), skip = shape, True
    print(f"[render {scene.config.name} {scene.config.width}x{scene.config.height}"
          f"x{scene.config.n_poses} mode={mode if shape is None else shape}]", flush=True)
    caches.set_lanes_per_ray(lanes)
    if centre > 0.0 and scene.config.sigma_channels == 0:
        caches.set_centre_block(centre)
    caches.set_empty_space_skipping(skip)
    P = torch.from_numpy(scene.poses if poses is None else poses).cuda()
    N = scene.config.n_samples if n_samples is None else n_samples
    try:
        if stats:
            rgb, depth, st = caches.render_stats(P, scene.intrinsics, scene.near, scene.far, N)
            rgb2, depth2 = caches.render(P, scene.intrinsics, scene.near, scene.far, N)
        else:
            rgb2, depth2 = caches.render(P, scene.intrinsics, scene.near, scene.far, N)
            rgb, depth, st = rgb2, depth2, None
        torch.cuda.synchronize()
        out = (rgb2.cpu().numpy().reshape(-1, 3), depth2.cpu().numpy().reshape(-1),
               None if st is None else st.cpu().numpy().view(np.uint32).reshape(-1, 4))
        if stats:
            # the diagnostics variant renders the same values
            assert np.array_equal(rgb.cpu().numpy().reshape(-1, 3), out[0])
            assert np.array_equal(depth.cpu().numpy().reshape(-1), out[1])
        return out
    finally:
        caches.close()


def compare(gpu, ref, ids, atol, label=""):
    """GPU outputs at ray ids vs oracle records: values within atol,
    stop / n_inbox / n_occ / hash bit-exact.  Returns the max errors."""
    rgb, depth, st = gpu
    e_rgb = float(np.max(np.abs(rgb[ids].astype(np.float64) - ref["rgb"]))) if len(ids) else 0.0
    e_dep = float(np.max(np.abs(depth[ids].astype(np.float64) - ref["depth"]))) if len(ids) else 0.0
    print(f"[parity {label}] rays={len(ids)} max|drgb|={e_rgb:.3g} max|ddepth|={e_dep:.3g}", flush=True)
    assert e_rgb <= atol, (label, e_rgb)
    assert e_dep <= atol, (label, e_dep)
    assert e_rgb <= REGRESSION_ATOL and e_dep <= REGRESSION_ATOL, (label, "regression bound", e_rgb, e_dep)
    if st is not None:
        s = st[ids]
        for k, name in enumerate(("stop", "n_inbox", "n_occ", "hash")):
            bad = np.nonzero(s[:, k] != ref[name])[0]
            assert bad.size == 0, (label, name, int(ids[bad[0]]), int(s[bad[0], k]), int(ref[name][bad[0]]))
    return e_rgb, e_dep


def sample_ray_ids(n_views, H, W, n_random, seed=0):
    """Random rays plus the image corners, edges and centre of each view."""
    rng = np.random.Generator(np.random.PCG64(seed))
    total = n_views * H * W
    ids = set(rng.integers(0, total, size=n_random).tolist())
    for b in range(n_views):
        base = b * H * W
        for v in (0, H // 2, H - 1):
            for u in (0, W // 2, W - 1):
                ids.add(base + v * W + u)
    return np.array(sorted(ids), dtype=np.int64)


class DeviceBuffer:
    """A raw hipMalloc allocation of exactly `nbytes` (torch's caching
    allocator hands out sub-ranges of larger segments, which hides
    undersized buffers from the library's range checks)."""

    def __init__(self, nbytes):
        import ctypes
        self._hip = ctypes.CDLL("libamdhip64.so")
        self.ptr = ctypes.c_void_p()
        rc = self._hip.hipMalloc(ctypes.byref(self.ptr), ctypes.c_size_t(nbytes))
        assert rc == 0, f"hipMalloc({nbytes}) failed: {rc}"

    def free(self):
        if self.ptr:
            self._hip.hipFree(self.ptr)
            self.ptr = None

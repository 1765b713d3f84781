"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Full frames at the small size; at the full workload sizes, sampled rays the
oracle renders one by one plus properties over the whole frame.  Values
within the stated tolerance, per-ray stop index, sample counts and the hash
of the occupied (i, ix, iy, iz) sequence bit-exact.
"""
import dataclasses
import math

import numpy as np
import pytest

import oracle
from paper_2204_02585_amd import scenes
from tests import parity_util as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2204_02585_amd import binding  # noqa: F401  (fails loudly without libsqn.so)


# ---------------------------------------------------------------- small sizes

MODES = list(pu.MODES)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("t_eps", [1e-4, 0.0])
def test_tiny_full_frame(t_eps, mode):
    sc = scenes.make_scene("tiny")
    gpu = pu.gpu_render(sc, t_eps=t_eps, mode=mode)
    ref = oracle.render_scene(sc, t_eps=t_eps)
    ids = np.arange(ref.size)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), f"tiny eps={t_eps} {mode}")
    assert (ref["n_occ"] > 0).sum() > 100


def _small(name, **kw):
    """A small variant of a named workload (same cache shape family)."""
    cfg = dataclasses.replace(scenes.CONFIGS[name], **kw)
    return scenes.make_scene(cfg)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("W,H", [(37, 23), (1, 1), (16, 16), (17, 1), (1, 33)])
def test_ragged_and_degenerate_image_sizes(W, H, mode):
    sc = _small("tiny", width=W, height=H, focal=1.25 * max(W, H))
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"{W}x{H}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("N", [1, 2, 3, 7, 384, 4096])
def test_sample_counts(N, mode):
    sc = _small("tiny", width=24, height=20, n_samples=N)
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"N={N}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("D", [1, 3, 8, 16, 32])
@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_component_counts_and_dtypes(D, dtype, mode):
    """Specialised (D = 8, 16) and generic kernels, both storage types."""
    sc = _small("tiny", width=40, height=40, D=D, dtype=dtype, n_p=48, n_theta=9, n_phi=12)
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"D={D} {dtype}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("sigma_dtype", ["f16", "f32"])
@pytest.mark.parametrize("n_p", [2, 5, 6, 7, 13, 50])
def test_plane_sizes_not_multiple_of_four(n_p, sigma_dtype, mode):
    """The packed sigma planes interleave four rows and pad the last group:
    plane sizes that are not a multiple of four, with one-word (binary16)
    and two-word (binary32) records.  At n_p = 2 no sample is occupied."""
    sc = _small("tiny", width=32, height=32, n_p=n_p, dtype="f16", sigma_dtype=sigma_dtype)
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"n_p={n_p} sigma {sigma_dtype}")
    assert (ref["n_occ"].sum() > 0) == (n_p > 2)


def test_paper_precision_mix():
    """sigma^j in fp32, u^j v^j w^j and beta in fp16 (Sec. 3.3)."""
    sc = _small("tiny", width=48, height=48)
    sc.uvw = [a.astype(np.float16) for a in sc.uvw]
    sc.beta = sc.beta.astype(np.float16)
    gpu = pu.gpu_render(sc)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), 1e-5, "sigma f32 / uvw f16")


@pytest.mark.parametrize("mode", MODES)
def test_stratified_small(mode):
    sc = _small("tiny", width=32, height=32, stratified=True)
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), "stratified")


@pytest.mark.parametrize("mode", MODES)
def test_multi_view_batch_small(mode):
    sc = _small("tiny", width=20, height=12)
    poses = scenes.spiral_poses(7)
    gpu = pu.gpu_render(sc, poses=poses, mode=mode)
    ref = oracle.render_scene(sc, poses=poses)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), "7 views")


@pytest.mark.parametrize("mode", MODES)
def test_camera_inside_box_and_axis_rays(mode):
    """Rays that start inside the box, run along box faces or have zero
    direction components (the clip's exact special case)."""
    sc = _small("tiny", width=9, height=9, focal=4.0)
    P = np.zeros((4, 3, 4), np.float32)
    # looking along +y from inside the box
    P[0, :, 0], P[0, :, 1], P[0, :, 2], P[0, :, 3] = (1, 0, 0), (0, 0, 1), (0, -1, 0), (0.1, -0.2, 0.3)
    # on the x = -1.5 face, looking along +y
    P[1, :, 0], P[1, :, 1], P[1, :, 2], P[1, :, 3] = (1, 0, 0), (0, 0, 1), (0, -1, 0), (-1.5, -4, 0.0)
    # on an edge (x = 1.5, z = -1.5), looking along +y
    P[2, :, 0], P[2, :, 1], P[2, :, 2], P[2, :, 3] = (1, 0, 0), (0, 0, 1), (0, -1, 0), (1.5, -4, -1.5)
    # looking straight down -z from above
    P[3, :, 0], P[3, :, 1], P[3, :, 2], P[3, :, 3] = (1, 0, 0), (0, 1, 0), (0, 0, 1), (0.2, 0.1, 4)
    gpu = pu.gpu_render(sc, poses=P, mode=mode)
    ref = oracle.render_scene(sc, poses=P)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), "inside/axis")
    assert ref["n_inbox"].sum() > 0


@pytest.mark.parametrize("name,mode", [("tiny", "skip1"), ("tiny", "skip4"), ("tiny", "skip8"),
                                       ("tiny_alt", "skip4")])
@pytest.mark.parametrize("stratified", [False, True])
@pytest.mark.parametrize("case", ["dense", "sparse", "far_camera", "near_zero"])
def test_leaps_land_past_empty_runs(case, stratified, name, mode):
    """A leap lands on the first sample past the run that a distance field
    (per plane, or the Eq. 5 cell grid) proves empty: no occupied sample may
    be skipped, with many samples per texel, several texels per sample, a
    large |near| / dt (the landing index's rounding slack) or near = 0."""
    radius, near, far, N = {"dense": (4.0, 2.0, 6.0, 2048), "sparse": (4.0, 2.0, 6.0, 24),
                            "far_camera": (60.0, 57.5, 62.5, 512), "near_zero": (4.0, 0.0, 8.0, 300)}[case]
    sc = _small(name, width=32, height=32, n_samples=N, focal=10.0 * radius, stratified=stratified)
    sc = dataclasses.replace(sc, near=near, far=far, poses=scenes.look_at_pose(radius, 45.0, 30.0)[None])
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"leaps {case}")
    assert ref["n_occ"].sum() > 0


@pytest.mark.parametrize("mode", MODES)
def test_dense_scene_terminates(mode):
    """sigma_max 2000: most rays stop within a few samples."""
    sc = _small("tiny", width=48, height=48, sigma_max=2000.0)
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), "dense")
    assert (ref["stop"] < sc.config.n_samples).mean() > 0.1


def test_two_streams_share_a_handle():
    """A handle is read-only while rendering, so renders on two streams may
    run at once: several rounds of concurrent launches on two side streams
    (default priority) give, bit for bit, the images of the same views
    rendered one after another on the current stream."""
    import torch
    from paper_2204_02585_amd import binding
    sc = _small("tiny", width=96, height=80, n_samples=96, focal=120.0)
    caches = binding.caches_from_scene(sc)
    try:
        pa = torch.from_numpy(scenes.spiral_poses(3)).cuda()
        pb = torch.from_numpy(scenes.spiral_poses(3, seed=5001)).cuda()
        ref_a = caches.render(pa, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        ref_b = caches.render(pb, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        torch.cuda.synchronize()
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        outs = []
        print("[two streams: 4 rounds of 2 concurrent renders]", flush=True)
        for _ in range(4):
            with torch.cuda.stream(s1):
                ra = caches.render(pa, sc.intrinsics, sc.near, sc.far, sc.config.n_samples, stream=s1)
            with torch.cuda.stream(s2):
                rb = caches.render(pb, sc.intrinsics, sc.near, sc.far, sc.config.n_samples, stream=s2)
            outs.append((ra, rb))
        torch.cuda.synchronize()
        for ra, rb in outs:
            for got, ref in ((ra, ref_a), (rb, ref_b)):
                assert torch.equal(got[0], ref[0]) and torch.equal(got[1], ref[1])
        assert float(ref_a[0].abs().sum()) > 0 and float(ref_b[0].abs().sum()) > 0
    finally:
        caches.close()


@pytest.mark.parametrize("mode", ["auto", "skip1", "L4"])
def test_depth_output_is_optional(mode):
    """depth_out may be NULL: the colours are those of a render with depth,
    bit for bit."""
    import torch
    from paper_2204_02585_amd import binding
    sc = _small("tiny", width=40, height=24)
    caches = binding.caches_from_scene(sc)
    try:
        lanes, skip = pu.MODES[mode]
        caches.set_lanes_per_ray(lanes)
        caches.set_empty_space_skipping(skip)
        P = torch.from_numpy(sc.poses).cuda()
        rgb, depth = caches.render(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        rgb2, none = caches.render(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples, with_depth=False)
        torch.cuda.synchronize()
        assert none is None
        assert torch.equal(rgb, rgb2)
        assert float(depth.max()) > 0
    finally:
        caches.close()


def test_empty_batch_is_noop():
    import torch
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny")
    caches = binding.caches_from_scene(sc)
    try:
        P = torch.zeros((0, 3, 4), device="cuda")
        rgb, depth = caches.render(P, sc.intrinsics, sc.near, sc.far, 64)
        torch.cuda.synchronize()
        assert rgb.shape == (0, 64, 64, 3)
    finally:
        caches.close()


def test_large_ragged_two_views():
    """Default launch on two 1000 x 700 views (not a multiple of the tile
    size) at a small sample count."""
    sc = _small("tiny", width=1000, height=700, n_samples=24, focal=1250.0)
    poses = scenes.spiral_poses(2)
    gpu = pu.gpu_render(sc, poses=poses, mode="auto")
    ref = oracle.render_scene(sc, poses=poses)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), "2x1000x700")
    assert (ref["n_occ"] > 0).sum() > 1000


# ------------------------------------------------------- full workload sizes

@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name,n_random", [("paper", 40000), ("large", 40000), ("paper512", 30000)])
def test_full_size_single_view(name, n_random, mode):
    sc = scenes.make_scene(name)
    cfg = sc.config
    gpu = pu.gpu_render(sc, mode=mode)
    ids = pu.sample_ray_ids(1, cfg.height, cfg.width, n_random, seed=cfg.number)
    ref = oracle.render_scene(sc, ray_ids=ids)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), name)
    rgb, depth, st = gpu
    # whole-frame properties
    assert np.all(rgb >= 0) and np.all(rgb <= 1.0 + 1e-6)
    assert np.all(depth >= 0) and np.all(depth <= sc.far + 1e-4)
    assert np.all(st[:, 0] <= cfg.n_samples) and np.all(st[:, 2] <= st[:, 1])


def test_full_size_batch():
    sc = scenes.make_scene("batch")
    cfg = sc.config
    gpu = pu.gpu_render(sc)
    ids = pu.sample_ray_ids(cfg.n_poses, cfg.height, cfg.width, 30000, seed=4)
    ref = oracle.render_scene(sc, ray_ids=ids)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), "batch")


@pytest.mark.parametrize("mode", ["auto", "skip1", "skip4", "L1"])
def test_full_size_stress(mode):
    sc = scenes.make_scene("stress")
    cfg = sc.config
    gpu = pu.gpu_render(sc, mode=mode)
    ids = pu.sample_ray_ids(1, cfg.height, cfg.width, 20000, seed=5)
    ref = oracle.render_scene(sc, ray_ids=ids)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), "stress")


@pytest.mark.parametrize("name,n_random", [("paper", 40000), ("large", 30000), ("paper512", 30000),
                                           ("stress", 20000), ("batch", 20000), ("llff", 20000)])
def test_full_size_recorded_launch_shapes(name, n_random):
    """Each workload in the launch shape bench.py times it in (its
    LAUNCH_SHAPES entry), sampled rays against the oracle."""
    import bench
    sc = scenes.make_scene(name)
    cfg = sc.config
    shape = bench.LAUNCH_SHAPES[name]
    gpu = pu.gpu_render(sc, shape=shape)
    ids = pu.sample_ray_ids(cfg.n_poses, cfg.height, cfg.width, n_random, seed=cfg.number)
    ref = oracle.render_scene(sc, ray_ids=ids)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), f"{name} shape {shape}")


# ------------------------------------------------------------ C-ABI errors

def test_abi_rejects_bad_arguments():
    import ctypes
    import torch
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny")
    caches = binding.caches_from_scene(sc)
    lib = binding.lib
    pose_buf = pu.DeviceBuffer(48)
    small = pu.DeviceBuffer(4096)
    try:
        P = torch.from_numpy(sc.poses).cuda()
        intr = binding.Intrinsics(80.0, 80.0, 32.0, 32.0, 64, 64)
        rgb = torch.empty((1, 64, 64, 3), device="cuda")
        h = caches.handle
        vp = ctypes.c_void_p

        def render(poses=vp(P.data_ptr()), n=1, intr_=ctypes.byref(intr), near=2.0, far=6.0,
                   N=64, out=vp(rgb.data_ptr()), depth=None):
            return lib.sqn_render(h, poses, n, intr_, near, far, N, out, depth, None)

        assert render() == binding.SQN_OK
        assert render(near=6.0, far=2.0) == binding.SQN_ERR_INVALID_ARG
        assert render(near=2.0, far=2.0) == binding.SQN_ERR_INVALID_ARG
        assert render(far=math.nan) == binding.SQN_ERR_INVALID_ARG
        assert render(N=0) == binding.SQN_ERR_INVALID_ARG
        assert render(N=40000) == binding.SQN_ERR_INVALID_ARG
        assert render(n=-1) == binding.SQN_ERR_INVALID_ARG
        # 100000 poses need 4.8 MB; this allocation holds one (allocation
        # granularity may round it up, but not to megabytes)
        assert render(poses=pose_buf.ptr, n=100000) == binding.SQN_ERR_INVALID_ARG
        assert "poses" in binding.last_error()
        # a 2048x2048 rgb image needs 48 MiB
        big = binding.Intrinsics(80.0, 80.0, 32.0, 32.0, 2048, 2048)
        assert render(intr_=ctypes.byref(big), out=small.ptr) == binding.SQN_ERR_INVALID_ARG
        assert "rgb_out" in binding.last_error()
        assert render(out=None) == binding.SQN_ERR_INVALID_ARG
        host = (ctypes.c_float * 12)()
        assert render(poses=ctypes.cast(host, vp)) == binding.SQN_ERR_INVALID_ARG
        assert render(intr_=None) == binding.SQN_ERR_INVALID_ARG
        bad = binding.Intrinsics(0.0, 80.0, 32.0, 32.0, 64, 64)
        assert render(intr_=ctypes.byref(bad)) == binding.SQN_ERR_INVALID_ARG
        empty = binding.Intrinsics(80.0, 80.0, 32.0, 32.0, 0, 64)
        assert render(intr_=ctypes.byref(empty)) == binding.SQN_ERR_INVALID_ARG
        assert lib.sqn_render(None, vp(P.data_ptr()), 1, ctypes.byref(intr), 2.0, 6.0, 64,
                              vp(rgb.data_ptr()), None, None) == binding.SQN_ERR_INVALID_ARG
        assert lib.sqn_render_stats(h, vp(P.data_ptr()), 1, ctypes.byref(intr), 2.0, 6.0, 64,
                                    vp(rgb.data_ptr()), None, None, None) == binding.SQN_ERR_INVALID_ARG
        torch.cuda.synchronize()
    finally:
        caches.close()
        pose_buf.free()
        small.free()
    lib.sqn_destroy(None)


def test_create_rejects_bad_descriptions_and_undersized_arrays():
    import ctypes
    import torch
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny")
    sig = [torch.from_numpy(a).cuda() for a in sc.sigma]
    uvw = [torch.from_numpy(a).cuda() for a in sc.uvw]
    beta = torch.from_numpy(sc.beta).cuda()
    with pytest.raises(binding.SqnError) as e:
        binding.Caches(sig, uvw, beta, (1, 1, 1), (-1, -1, -1))
    assert e.value.status == binding.SQN_ERR_INVALID_ARG
    with pytest.raises(binding.SqnError) as e:
        binding.Caches(sig, uvw, beta, sc.bbox_min, sc.bbox_max, t_eps=2.0)
    assert e.value.status == binding.SQN_ERR_INVALID_ARG
    # n_p = 2048 needs 16 MiB sigma planes and 384 MiB uvw planes; the
    # arrays given are far smaller
    short = pu.DeviceBuffer(4096)
    try:
        desc = binding.CacheDesc()
        desc.n_p, desc.D, desc.n_theta, desc.n_phi = 2048, 8, 32, 32
        for r in range(3):
            desc.bbox_min[r], desc.bbox_max[r] = -1.5, 1.5
        desc.t_eps = 1e-4
        vp = ctypes.c_void_p
        sp = (vp * 3)(*[s.data_ptr() for s in sig])
        up = (vp * 3)(uvw[0].data_ptr(), short.ptr.value, uvw[2].data_ptr())
        out = vp()
        rc = binding.lib.sqn_create_caches(ctypes.byref(desc), sp, up, vp(beta.data_ptr()), None,
                                           ctypes.byref(out))
        assert rc == binding.SQN_ERR_INVALID_ARG and not out
        assert "sigma_planes[0]" in binding.last_error()
        desc.D = 33
        up = (vp * 3)(*[u.data_ptr() for u in uvw])
        assert binding.lib.sqn_create_caches(ctypes.byref(desc), sp, up, vp(beta.data_ptr()), None,
                                             ctypes.byref(out)) == binding.SQN_ERR_INVALID_ARG
    finally:
        short.free()


def test_launch_option_validation():
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny")
    caches = binding.caches_from_scene(sc)
    try:
        for bad in (2, 3, -1, 16):
            with pytest.raises(binding.SqnError):
                caches.set_lanes_per_ray(bad)
        for good in (0, 1, 4, 8):
            caches.set_lanes_per_ray(good)
        for bad in (2, -1):
            assert binding.lib.sqn_set_empty_space_skipping(caches.handle, bad) == binding.SQN_ERR_INVALID_ARG
        caches.set_empty_space_skipping(False)
        caches.set_empty_space_skipping(True)
    finally:
        caches.close()
    assert binding.lib.sqn_set_lanes_per_ray(None, 1) == binding.SQN_ERR_INVALID_ARG
    assert binding.lib.sqn_set_empty_space_skipping(None, 1) == binding.SQN_ERR_INVALID_ARG


@pytest.mark.parametrize("fraction", [0.15, 0.5, 1.0])
@pytest.mark.parametrize("W,H", [(1, 1), (37, 23), (16, 16), (70, 33), (64, 64)])
def test_hybrid_launch_fractions(W, H, fraction):
    """Hybrid launches: the centred rectangle of 16-pixel blocks with four
    lanes per ray (all of the image at fraction 1), the rest with one, at
    ragged image sizes; the stats variant renders the same values."""
    import torch
    from paper_2204_02585_amd import binding
    sc = _small("tiny", width=W, height=H, focal=1.25 * max(W, H))
    caches = binding.caches_from_scene(sc)
    try:
        caches.set_centre_block(fraction)
        P = torch.from_numpy(sc.poses).cuda()
        rgb, depth, st = caches.render_stats(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        rgb2, depth2 = caches.render(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        torch.cuda.synchronize()
        assert torch.equal(rgb, rgb2) and torch.equal(depth, depth2)
        gpu = (rgb2.cpu().numpy().reshape(-1, 3), depth2.cpu().numpy().reshape(-1),
               st.cpu().numpy().view(np.uint32).reshape(-1, 4))
        ref = oracle.render_scene(sc)
        pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"hybrid {fraction} {W}x{H}")
        for bad in (-0.1, 1.5, float("nan")):
            with pytest.raises(binding.SqnError):
                caches.set_centre_block(bad)
    finally:
        caches.close()


@pytest.mark.parametrize("views", [1, 3])
def test_tune_lanes_per_ray(views):
    """sqn_tune_lanes_per_ray picks one of the launch shapes by timing them
    on the batch; renders after it (one lane per ray on a single view deals
    its tiles from the centre outwards) keep parity with the oracle."""
    import torch
    from paper_2204_02585_amd import binding
    sc = _small("tiny", width=48, height=40, n_poses=views)
    caches = binding.caches_from_scene(sc)
    try:
        P = torch.from_numpy(sc.poses).cuda()
        chosen = caches.tune_lanes_per_ray(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        assert chosen in ((-1, 1, 4, 8) if views == 1 else (1, 4, 8))
        rgb, depth = caches.render(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples)
        torch.cuda.synchronize()
        gpu = (rgb.cpu().numpy().reshape(-1, 3), depth.cpu().numpy().reshape(-1), None)
        ref = oracle.render_scene(sc)
        pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"tuned L={chosen} views={views}")
        # a bad batch leaves the handle as it was and reports the error
        bad = binding.lib.sqn_tune_lanes_per_ray(caches.handle, binding._ptr(P), views, None, sc.near, sc.far,
                                                 sc.config.n_samples, None, None, None, None, None)
        assert bad == binding.SQN_ERR_INVALID_ARG
    finally:
        caches.close()
    assert binding.lib.sqn_tune_lanes_per_ray(None, None, 0, None, 2.0, 6.0, 1, None, None, None,
                                              None, None) == binding.SQN_ERR_INVALID_ARG


def test_create_out_of_memory_hook(monkeypatch):
    import torch
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny")
    monkeypatch.setenv("SQN_TEST_FAIL_ALLOC", "1")
    free0 = torch.cuda.mem_get_info()[0]
    with pytest.raises(binding.SqnError) as e:
        binding.caches_from_scene(sc)
    assert e.value.status == binding.SQN_ERR_OUT_OF_MEMORY
    monkeypatch.delenv("SQN_TEST_FAIL_ALLOC")
    c = binding.caches_from_scene(sc)
    assert c.device_bytes >= sc.cache_nbytes()
    c.close()
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] >= free0 - (64 << 20)

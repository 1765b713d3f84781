"""GPU parity of the Eq. 5 ("SqueezeNeRF (alt)") decoder: the HIP path
through sqn_create_linear_caches against the CPU oracle's literal Eq. 5.

Same contract as the Eq. 4 tests: values within the stated tolerance;
per-ray stop index, sample counts and the hash of the occupied
(i, ix, iy, iz) sequence bit-exact (the density is evaluated in the same
binary32 order on both sides).
"""
import ctypes
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2204_02585_amd import scenes
from tests import parity_util as pu

pytestmark = pytest.mark.gpu

# the linear decoder always renders with four lanes per ray
MODES = ["auto", "skip4", "L4"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2204_02585_amd import binding  # noqa: F401  (fails loudly without libsqn.so)


def _small(**kw):
    return scenes.make_scene(dataclasses.replace(scenes.CONFIGS["tiny_alt"], **kw))


def _full_frame(sc, mode, label, t_eps=None):
    gpu = pu.gpu_render(sc, t_eps=t_eps, mode=mode)
    ref = oracle.render_scene(sc, t_eps=t_eps)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), label)
    return ref


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("t_eps", [1e-4, 0.0])
def test_tiny_alt_full_frame(t_eps, mode):
    sc = scenes.make_scene("tiny_alt")
    ref = _full_frame(sc, mode, f"tiny_alt eps={t_eps} {mode}", t_eps=t_eps)
    assert (ref["n_occ"] > 0).sum() > 500
    if t_eps > 0:
        assert (ref["stop"] < sc.config.n_samples).sum() > 100


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("D", [1, 3, 8, 16])
@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_alt_component_counts_and_dtypes(D, dtype, mode):
    sc = _small(D=D, dtype=dtype, width=40, height=24, focal=50.0)
    _full_frame(sc, mode, f"alt D={D} {dtype} {mode}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("n_p", [6, 7, 13, 50])
def test_alt_plane_sizes_not_multiple_of_four(n_p, mode):
    """The Eq. 5 planes are moved into the four-row interleaved order at
    creation, the last group of rows padded."""
    sc = _small(n_p=n_p, width=32, height=24, focal=40.0)
    ref = _full_frame(sc, mode, f"alt n_p={n_p} {mode}")
    assert ref["n_occ"].sum() > 0


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("d_sigma", [1, 5, 64])
def test_alt_density_channel_counts(d_sigma, mode):
    sc = _small(sigma_channels=d_sigma, width=40, height=24, focal=50.0)
    _full_frame(sc, mode, f"alt d_sigma={d_sigma} {mode}")


@pytest.mark.parametrize("mode", MODES)
def test_alt_signed_density_weights(mode):
    """Mixed-sign W_sigma and a bias near the features' range: the density
    is irregular, and the empty-texel bound must use the row and column
    maxima of the other planes."""
    sc = scenes.make_scene("tiny_alt")
    rng = np.random.Generator(np.random.PCG64(77))
    dec = sc.decoder
    scale = float(np.max(dec.w_sigma))
    sc.decoder = scenes.LinearDecoder(
        (scale * rng.uniform(-1.0, 1.0, size=dec.w_sigma.size)).astype(np.float32),
        float(np.float32(-0.6 * scale)), dec.w_uvw, dec.b_uvw)
    ref = _full_frame(sc, mode, f"alt signed {mode}")
    assert (ref["n_occ"] > 0).sum() > 100


@pytest.mark.parametrize("mode", MODES)
def test_alt_stratified_multi_view(mode):
    sc = _small(n_poses=3, stratified=True, width=33, height=20, focal=45.0)
    sc.poses = scenes.spiral_poses(3)
    _full_frame(sc, mode, f"alt stratified x3 {mode}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("N", [1, 7, 384])
def test_alt_sample_counts(N, mode):
    sc = _small(n_samples=N, width=24, height=24, focal=30.0)
    _full_frame(sc, mode, f"alt N={N} {mode}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name,n_random", [("alt", 40000), ("alt512", 20000)])
def test_alt_full_size_single_view(name, n_random, mode):
    sc = scenes.make_scene(name)
    cfg = sc.config
    gpu = pu.gpu_render(sc, mode=mode)
    ids = pu.sample_ray_ids(1, cfg.height, cfg.width, n_random, seed=cfg.number)
    ref = oracle.render_scene(sc, ray_ids=ids)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), f"{name} {mode}")
    rgb, depth, st = gpu
    assert np.all(rgb >= 0) and np.all(rgb <= 1.0 + 1e-6)
    assert np.all(depth >= 0) and np.all(depth <= sc.far + 1e-4)
    assert np.all(st[:, 0] <= cfg.n_samples) and np.all(st[:, 2] <= st[:, 1])


def test_alt_batch_of_views():
    """More than 2^20 rays (where Eq. 4 handles switch to one lane per ray)."""
    sc = scenes.make_scene(dataclasses.replace(scenes.CONFIGS["alt"], n_poses=3))
    sc.poses = scenes.spiral_poses(3)
    cfg = sc.config
    gpu = pu.gpu_render(sc)
    ids = pu.sample_ray_ids(3, cfg.height, cfg.width, 20000, seed=11)
    ref = oracle.render_scene(sc, ray_ids=ids)
    pu.compare(gpu, ref, ids, pu.scene_atol(sc), "alt x3")


# ------------------------------------------------------------ C-ABI errors

def test_linear_create_rejects_bad_decoders():
    import torch
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny_alt")
    sig = [torch.from_numpy(a).cuda() for a in sc.sigma]
    uvw = [torch.from_numpy(a).cuda() for a in sc.uvw]
    beta = torch.from_numpy(sc.beta).cuda()
    dec = sc.decoder
    D = sc.config.D

    good_desc = _desc_of(sc, sig, uvw, beta, dec)

    def create(decoder_struct, sigma_ptrs=None, desc=good_desc):
        vp = ctypes.c_void_p
        sp = (vp * 3)(*(sigma_ptrs or [s.data_ptr() for s in sig]))
        up = (vp * 3)(*[u.data_ptr() for u in uvw])
        out = vp()
        rc = binding.lib.sqn_create_linear_caches(ctypes.byref(desc), decoder_struct, sp, up,
                                                  vp(beta.data_ptr()), None, ctypes.byref(out))
        if out:
            binding.lib.sqn_destroy(out)
        return rc, bool(out)

    w_s = np.array(dec.w_sigma, np.float32)
    w_u = np.array(dec.w_uvw, np.float32)
    b_u = np.array(dec.b_uvw, np.float32)

    def struct(ds=12, b=dec.b_sigma, ws=w_s, wu=w_u, bu=b_u):
        return ctypes.byref(binding.LinearDecoder(ds, b, None if ws is None else ws.ctypes.data,
                                                  None if wu is None else wu.ctypes.data,
                                                  None if bu is None else bu.ctypes.data))

    assert create(struct()) == (binding.SQN_OK, True)
    assert create(None) == (binding.SQN_ERR_INVALID_ARG, False)
    for bad in (struct(ds=0), struct(ds=65), struct(b=float("nan")), struct(ws=None),
                struct(wu=None), struct(bu=None)):
        assert create(bad) == (binding.SQN_ERR_INVALID_ARG, False)
    for arr in (w_s, w_u, b_u):
        keep = arr.flat[1]
        arr.flat[1] = np.inf
        assert create(struct()) == (binding.SQN_ERR_INVALID_ARG, False)
        assert "not finite" in binding.last_error()
        arr.flat[1] = keep
    # n_p = 1024 with 12 channels needs 48 MiB per sigma plane; the
    # buffers given hold 4 KiB (raw allocations: torch's segments would hide
    # the shortfall)
    short = pu.DeviceBuffer(4096)
    try:
        desc = _desc_of(sc, sig, uvw, beta, dec)
        desc.n_p = 1024
        assert desc.n_p != good_desc.n_p
        rc = create(struct(), sigma_ptrs=[short.ptr.value] * 3, desc=desc)
        assert rc == (binding.SQN_ERR_INVALID_ARG, False)
        assert "sigma_planes[0]" in binding.last_error()
    finally:
        short.free()
    assert D == 8


def _desc_of(sc, sig, uvw, beta, dec):
    from paper_2204_02585_amd import binding
    c = binding.Caches(sig, uvw, beta, sc.bbox_min, sc.bbox_max, decoder=dec)
    desc = c.desc
    c.close()
    return desc


def test_linear_tune_keeps_four_lanes():
    """The linear decoder renders with four lanes per ray only, so tuning
    measures that one shape and keeps it."""
    import torch
    from paper_2204_02585_amd import binding
    sc = _small(width=32, height=24, focal=40.0)
    caches = binding.caches_from_scene(sc)
    try:
        P = torch.from_numpy(sc.poses).cuda()
        assert caches.tune_lanes_per_ray(P, sc.intrinsics, sc.near, sc.far, sc.config.n_samples) == 4
        with pytest.raises(binding.SqnError):
            caches.set_centre_block(0.5)
        caches.set_centre_block(0.0)
    finally:
        caches.close()


def test_linear_handle_options():
    from paper_2204_02585_amd import binding
    sc = scenes.make_scene("tiny_alt")
    caches = binding.caches_from_scene(sc)
    try:
        for other in (1, 8):
            with pytest.raises(binding.SqnError) as e:
                caches.set_lanes_per_ray(other)
            assert e.value.status == binding.SQN_ERR_UNSUPPORTED
        caches.set_lanes_per_ray(4)
        caches.set_lanes_per_ray(0)
        caches.set_empty_space_skipping(False)
        caches.set_empty_space_skipping(True)
        # partial-sum records (8 B per texel) replace the 12-channel planes
        n_p, D = sc.config.n_p, sc.config.D
        assert caches.device_bytes >= 3 * n_p * n_p * (8 + 3 * D * 4)
    finally:
        caches.close()

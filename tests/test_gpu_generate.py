"""GPU parity of cache generation (sqn_create_networks / sqn_generate_caches)
against the binary64 oracle (oracle/cachegen.py).

Tolerance: the GPU multiplies binary16 weights by binary16 activations with
binary32 accumulation, rounding every hidden activation and the encoding to
binary16 (relative 2^-11 each) through up to 7 layers, then stores uvw and
beta as binary16.  Emulating exactly that rounding in binary64 gives at most
2.5e-3 (1 + |x|) on the synthetic networks; the bar is 1e-2 (1 + |x|).
"""
import dataclasses

import numpy as np
import pytest

from oracle import cachegen as cg
from paper_2204_02585_amd import scenes

pytestmark = pytest.mark.gpu

REL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2204_02585_amd import binding  # noqa: F401


def _check(got, want, label):
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - want) / (1.0 + np.abs(want))
    print(f"[generate {label}] n={want.size} max rel err {err.max():.3g} max|x| {np.abs(want).max():.3g}",
          flush=True)
    assert err.max() <= REL, (label, float(err.max()))


def _generate(g, n_p=None, n_theta=None, n_phi=None, dtypes=("f32", "f32", "f32")):
    import torch
    from paper_2204_02585_amd import binding
    c = g.config
    n_p = c.n_p if n_p is None else n_p
    n_theta = c.n_theta if n_theta is None else n_theta
    n_phi = c.n_phi if n_phi is None else n_phi
    tmap = {"f32": torch.float32, "f16": torch.float16}
    print(f"[generate {c.name} n_p={n_p} dirs={n_theta}x{n_phi} dtypes={dtypes}]", flush=True)
    nets = binding.networks_from_gen_scene(g)
    try:
        sig, uvw, beta = nets.generate(n_p, n_theta, n_phi, g.bbox_min, g.bbox_max, *[tmap[d] for d in dtypes])
        torch.cuda.synchronize()
        return ([s.float().cpu().numpy() for s in sig], [u.float().cpu().numpy() for u in uvw],
                beta.float().cpu().numpy())
    finally:
        nets.close()


def _full_compare(g, label, **kw):
    c = g.config
    n_p = kw.get("n_p", c.n_p)
    n_theta, n_phi = kw.get("n_theta", c.n_theta), kw.get("n_phi", c.n_phi)
    sig, uvw, beta = _generate(g, **kw)
    rs, ru, rb = cg.caches(g.pos, g.dir, n_p, n_theta, n_phi, g.bbox_min, g.bbox_max, c.D,
                           c.pos_freq, c.dir_freq)
    for j in range(3):
        _check(sig[j], rs[j], f"{label} sigma[{j}]")
        _check(uvw[j], ru[j], f"{label} uvw[{j}]")
    _check(beta, rb, f"{label} beta")


def test_generate_tiny_full_grids():
    _full_compare(scenes.make_gen_scene("gen_tiny"), "tiny")


@pytest.mark.parametrize("dtypes", [("f32", "f16", "f16"), ("f16", "f16", "f16")])
def test_generate_tiny_storage_dtypes(dtypes):
    _full_compare(scenes.make_gen_scene("gen_tiny"), f"tiny {dtypes}", dtypes=dtypes)


@pytest.mark.parametrize("n_p,n_theta,n_phi", [(2, 2, 2), (37, 5, 7), (129, 3, 130)])
def test_generate_ragged_grids(n_p, n_theta, n_phi):
    _full_compare(scenes.make_gen_scene("gen_tiny"), f"ragged {n_p}", n_p=n_p, n_theta=n_theta, n_phi=n_phi)


@pytest.mark.parametrize("kw", [dict(D=1), dict(D=3), dict(D=16), dict(D=32),
                                dict(pos_layers=1, dir_layers=1), dict(pos_layers=9, dir_layers=2),
                                dict(pos_freq=0, dir_freq=0), dict(pos_freq=15, dir_freq=10)])
def test_generate_network_shapes(kw):
    cfg = dataclasses.replace(scenes.GEN_CONFIGS["gen_tiny"], n_p=24, **kw)
    _full_compare(scenes.make_gen_scene(cfg), f"shape {kw}")


@pytest.mark.parametrize("name", ["gen_512", "gen_1k"])
def test_generate_full_size_sampled(name):
    """The paper's 512 and 1K grids: sampled texels of every plane against
    the oracle evaluated at those points only, all direction nodes."""
    g = scenes.make_gen_scene(name)
    c = g.config
    sig, uvw, beta = _generate(g, dtypes=("f32", "f16", "f16"))
    rng = np.random.Generator(np.random.PCG64(c.number))
    for j in range(3):
        ia = np.concatenate([[0, c.n_p - 1, 0, c.n_p - 1], rng.integers(0, c.n_p, 3000)])
        ib = np.concatenate([[0, 0, c.n_p - 1, c.n_p - 1], rng.integers(0, c.n_p, 3000)])
        rs, ru = cg.position_cache_points(g.pos[j], c.n_p, j, g.bbox_min, g.bbox_max, c.D, ia, ib, c.pos_freq)
        _check(sig[j][ia, ib], rs, f"{name} sigma[{j}]")
        _check(uvw[j][ia, ib], ru, f"{name} uvw[{j}]")
        assert np.all(np.isfinite(sig[j])) and np.all(np.isfinite(uvw[j]))
    _check(beta, cg.direction_cache(g.dir, c.n_theta, c.n_phi, c.dir_freq), f"{name} beta")


def test_generated_caches_render():
    """The generated arrays are accepted by sqn_create_caches and render."""
    import torch
    from paper_2204_02585_amd import binding
    g = scenes.make_gen_scene("gen_tiny")
    c = g.config
    nets = binding.networks_from_gen_scene(g)
    try:
        sig, uvw, beta = nets.generate(c.n_p, c.n_theta, c.n_phi, g.bbox_min, g.bbox_max)
        caches = binding.Caches(sig, uvw, beta, g.bbox_min, g.bbox_max)
        pose = torch.from_numpy(scenes.single_pose()).cuda()
        intr = dict(fx=40.0, fy=40.0, cx=16.0, cy=16.0, width=32, height=32)
        rgb, depth = caches.render(pose, intr, 2.0, 6.0, 64)
        torch.cuda.synchronize()
        assert torch.isfinite(rgb).all() and (rgb >= 0).all() and (rgb <= 1).all()
        caches.close()
    finally:
        nets.close()


def test_network_validation():
    import torch
    from paper_2204_02585_amd import binding
    g = scenes.make_gen_scene("gen_tiny")
    c = g.config
    with pytest.raises(binding.SqnError) as e:
        binding.Networks(g.pos, g.dir, c.D + 1)          # head sizes do not match D
    assert e.value.status == binding.SQN_ERR_INVALID_ARG
    with pytest.raises(binding.SqnError) as e:
        binding.Networks(g.pos, g.dir, c.D, pos_freq=9)  # 42 inputs given, 38 expected
    assert e.value.status == binding.SQN_ERR_INVALID_ARG
    bad = [list(l) for l in g.pos]
    W = bad[1][2][0].copy()
    W[3, 4] = np.float16(np.inf)
    bad[1][2] = (W, bad[1][2][1])
    with pytest.raises(binding.SqnError) as e:
        binding.Networks(bad, g.dir, c.D)
    assert "not finite" in str(e.value)
    narrow = scenes.mlp_weights([c.pos_in, 128, 128, c.pos_out], 1)     # 128-unit position networks
    with pytest.raises(binding.SqnError) as e:
        binding.Networks([narrow] * 3, g.dir, c.D)
    assert e.value.status == binding.SQN_ERR_UNSUPPORTED
    nets = binding.networks_from_gen_scene(g)
    try:
        assert nets.device_bytes > 0
        # outputs too small for the requested grid (raw allocations: torch's
        # segments would hide the shortfall)
        from tests import parity_util as pu
        small = pu.DeviceBuffer(4096)
        try:
            import ctypes
            desc = binding.CacheDesc()
            desc.n_p, desc.D, desc.n_theta, desc.n_phi = 512, c.D, 8, 8
            for r in range(3):
                desc.bbox_min[r], desc.bbox_max[r] = -1.5, 1.5
            vp = ctypes.c_void_p
            beta = torch.empty((8, 8, c.D), device="cuda")
            ptrs = (vp * 3)(*([small.ptr.value] * 3))
            rc = binding.lib.sqn_generate_caches(nets.handle, ctypes.byref(desc), ptrs, ptrs,
                                                 vp(beta.data_ptr()), None)
            assert rc == binding.SQN_ERR_INVALID_ARG and "sigma_planes[0]" in binding.last_error()
            desc.D = c.D + 1
            rc = binding.lib.sqn_generate_caches(nets.handle, ctypes.byref(desc), ptrs, ptrs,
                                                 vp(beta.data_ptr()), None)
            assert rc == binding.SQN_ERR_INVALID_ARG and "D" in binding.last_error()
        finally:
            small.free()
    finally:
        nets.close()
    assert binding.lib.sqn_generate_caches(None, None, None, None, None, None) == binding.SQN_ERR_INVALID_ARG
    binding.lib.sqn_destroy_networks(None)


def draw_gen_case(k):
    """Generation case k from a generator seeded by k: grid sizes, D, depth
    of both networks, encoding frequencies and the three storage types."""
    rng = np.random.Generator(np.random.PCG64(9000 + k))
    cfg = dataclasses.replace(
        scenes.GEN_CONFIGS["gen_tiny"], name=f"gen_rand{k}", number=200 + k,
        n_p=int(rng.integers(2, 81)), n_theta=int(rng.integers(2, 41)), n_phi=int(rng.integers(2, 41)),
        D=int(rng.integers(1, 33)), pos_layers=int(rng.integers(1, 9)), dir_layers=int(rng.integers(1, 6)),
        pos_freq=int(rng.integers(0, 13)), dir_freq=int(rng.integers(0, 7)))
    dtypes = tuple(("f32", "f16")[int(rng.integers(0, 2))] for _ in range(3))
    return cfg, dtypes


@pytest.mark.parametrize("k", range(24))
def test_generate_random_configurations(k):
    """Seeded random combinations of grid sizes, D, network depths,
    encoding frequencies and storage types, whole grids against the
    oracle."""
    cfg, dtypes = draw_gen_case(k)
    g = scenes.make_gen_scene(cfg)
    _full_compare(g, f"random {k} D={cfg.D} layers={cfg.pos_layers}/{cfg.dir_layers} "
                     f"freq={cfg.pos_freq}/{cfg.dir_freq} {dtypes}", dtypes=dtypes)

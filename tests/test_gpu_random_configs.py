"""GPU parity on seeded random combinations of every option at once.

The other parity tests vary one option at a time; here each case draws an
image size, sample count, plane size, D, storage types, direction grid,
density scale, views, stratified sampling, termination threshold, decoder
(Eq. 4 or Eq. 5), world or NDC rays and launch shape together, and the whole
frame is compared with the oracle: values within the tolerance of the cache
dtype (and the regression bound), stop index, sample counts and the hash of
the occupied (i, ix, iy, iz) sequence bit for bit.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2204_02585_amd import scenes
from tests import parity_util as pu

pytestmark = pytest.mark.gpu

N_CASES = 150


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2204_02585_amd import binding  # noqa: F401  (fails loudly without libsqn.so)


def draw_case(k):
    """Case k: a Config and a launch mode, from a generator seeded by k."""
    rng = np.random.Generator(np.random.PCG64(7000 + k))
    base = ("tiny", "tiny", "tiny_alt", "llff_tiny")[int(rng.integers(0, 4))]
    cfg = scenes.CONFIGS[base]
    W, H = int(rng.integers(1, 73)), int(rng.integers(1, 73))
    dtype = ("f32", "f16")[int(rng.integers(0, 2))]
    over = dict(
        name=f"rand{k}", number=100 + k, width=W, height=H,
        n_samples=int(np.exp(rng.uniform(0.0, np.log(320.0)))),
        n_p=int(rng.integers(2, 97)),
        D=int((1, 2, 3, 5, 8, 8, 16, 16)[int(rng.integers(0, 8))]),
        n_theta=int(rng.integers(2, 41)), n_phi=int(rng.integers(2, 41)),
        dtype=dtype, sigma_dtype=(None, "f32", "f16")[int(rng.integers(0, 3))],
        n_blobs=int(rng.integers(1, 33)),
        sigma_max=float((5.0, 50.0, 500.0)[int(rng.integers(0, 3))]),
        stratified=bool(rng.integers(0, 2)),
        t_eps=float((0.0, 1e-4, 1e-2)[int(rng.integers(0, 3))]),
        n_poses=int((1, 1, 2, 3)[int(rng.integers(0, 4))]),
    )
    if not cfg.forward:
        over["focal"] = 1.25 * max(W, H)
    if cfg.sigma_channels > 0:
        over["sigma_channels"] = int(rng.integers(1, 17))
    cfg = dataclasses.replace(cfg, **over)
    if cfg.sigma_channels > 0:
        modes = ["auto", "skip4", "L4"]          # the linear decoder runs four lanes per ray
    else:
        modes = list(pu.MODES)
    mode = modes[int(rng.integers(0, len(modes)))]
    return cfg, mode


@pytest.mark.parametrize("k", range(N_CASES))
def test_random_configuration_full_frame(k):
    cfg, mode = draw_case(k)
    print(f"[random case {k}: {cfg.width}x{cfg.height}x{cfg.n_poses} N={cfg.n_samples} n_p={cfg.n_p} "
          f"D={cfg.D} {cfg.dtype}/{cfg.sigma_dtype} dir={cfg.n_theta}x{cfg.n_phi} blobs={cfg.n_blobs} "
          f"smax={cfg.sigma_max} strat={cfg.stratified} eps={cfg.t_eps} d_sigma={cfg.sigma_channels} "
          f"ndc={cfg.forward} mode={mode}]", flush=True)
    sc = scenes.make_scene(cfg)
    gpu = pu.gpu_render(sc, mode=mode)
    ref = oracle.render_scene(sc)
    pu.compare(gpu, ref, np.arange(ref.size), pu.scene_atol(sc), f"random {k} {mode}")

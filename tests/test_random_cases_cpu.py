"""The random GPU parity cases (tests/test_gpu_random_configs.py) are drawn
from seeded generators; this checks on the CPU that they reach every option
the renderer has and that the oracle renders each of them."""
import numpy as np

import oracle
from paper_2204_02585_amd import scenes
from tests.test_gpu_random_configs import N_CASES, draw_case


def test_cases_cover_the_options():
    """The drawn cases reach every decoder, ray model, storage type, launch
    mode and a spread of sizes (checked without a GPU run of them)."""
    cases = [draw_case(k) for k in range(N_CASES)]
    cfgs = [c for c, _ in cases]
    assert any(c.sigma_channels > 0 for c in cfgs) and any(c.forward for c in cfgs)
    assert any(c.sigma_channels == 0 and not c.forward for c in cfgs)
    assert {c.dtype for c in cfgs} == {"f32", "f16"}
    assert {c.D for c in cfgs} >= {8, 16} and any(c.D not in (8, 16) for c in cfgs)
    assert any(c.stratified for c in cfgs) and any(c.t_eps == 0.0 for c in cfgs)
    assert any(c.n_poses > 1 for c in cfgs)
    assert len({m for _, m in cases}) >= 6
    assert any(c.n_p % 4 != 0 for c in cfgs) and any(c.width * c.height < 64 for c in cfgs)


def test_oracle_renders_every_case():
    """Every drawn case builds and the oracle renders it (the GPU side is
    compared with this in the GPU test); some rays of some cases see
    occupied samples and some stop early."""
    occupied = stopped = 0
    for k in range(N_CASES):
        cfg, _ = draw_case(k)
        sc = scenes.make_scene(cfg)
        ref = oracle.render_scene(sc)
        assert ref.size == cfg.width * cfg.height * cfg.n_poses
        assert np.all(np.isfinite(ref["rgb"])) and np.all(np.isfinite(ref["depth"]))
        occupied += int((ref["n_occ"] > 0).sum())
        stopped += int((ref["stop"] < cfg.n_samples).sum())
    assert occupied > 1000 and stopped > 100

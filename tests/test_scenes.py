"""The seeded input generator: shapes, determinism, and the separable blob."""
import math

import numpy as np

from paper_2204_02585_amd import scenes


def test_single_blob_is_exactly_separable():
    """exp(-|d|^2 / 2s^2) = prod over the planes xy, yz, zx of
    exp(-(da^2 + db^2) / 4s^2), because each axis appears in two planes; so
    the product rule of Eq. 4 reproduces a 3-D Gaussian blob at every node
    where all three planar factors are inside their cut-off."""
    n_p = 33
    blobs = scenes.Blobs(np.array([[0.1, -0.2, 0.3]]), np.array([1.0]), 27.0)
    sxy, syz, szx = scenes.bake_sigma_planes(n_p, blobs, np.float64)
    x = scenes.node_coords(n_p, -1.5, 1.5)
    s, rho = 0.25, 0.6
    c = blobs.centre[0]
    checked = 0
    for a in range(n_p):
        for b in range(n_p):
            for k in range(n_p):
                pxy = (x[a] - c[0]) ** 2 + (x[b] - c[1]) ** 2
                pyz = (x[b] - c[1]) ** 2 + (x[k] - c[2]) ** 2
                pzx = (x[k] - c[2]) ** 2 + (x[a] - c[0]) ** 2
                got = sxy[a, b] * syz[b, k] * szx[k, a]
                if max(pxy, pyz, pzx) <= rho * rho:
                    r2 = (x[a] - c[0]) ** 2 + (x[b] - c[1]) ** 2 + (x[k] - c[2]) ** 2
                    want = 27.0 * math.exp(-r2 / (2 * s * s))
                    assert abs(got - want) <= 1e-12 * 27.0
                    checked += 1
                else:
                    assert got == 0.0
    assert checked > 10


def test_configs_shapes_and_determinism():
    a = scenes.make_scene("tiny")
    b = scenes.make_scene("tiny")
    cfg = a.config
    assert [p.shape for p in a.sigma] == [(64, 64)] * 3
    assert [p.shape for p in a.uvw] == [(64, 64, 24)] * 3
    assert a.beta.shape == (32, 32, 8) and a.poses.shape == (1, 3, 4)
    assert all(p.dtype == np.float32 for p in a.sigma + a.uvw)
    for x, y in zip(a.sigma + a.uvw + [a.beta, a.poses], b.sigma + b.uvw + [b.beta, b.poses]):
        assert np.array_equal(x, y)
    assert cfg.fx == 80.0 and a.intrinsics["cx"] == 32.0
    assert a.cache_nbytes() == 3 * 64 * 64 * (4 + 24 * 4) + 32 * 32 * 8 * 4


def test_pose_is_a_rotation_looking_at_origin():
    P = scenes.look_at_pose(4.0, 45.0, 30.0).astype(np.float64)
    R, c = P[:, :3], P[:, 3]
    assert np.allclose(R.T @ R, np.eye(3), atol=1e-6)
    assert np.allclose(np.linalg.det(R), 1.0, atol=1e-6)
    assert np.allclose(-R[:, 2], -c / np.linalg.norm(c), atol=1e-6)   # looks at the origin
    assert abs(np.linalg.norm(c) - 4.0) < 1e-5


def test_spiral_poses_ranges():
    P = scenes.spiral_poses(100).astype(np.float64)
    r = np.linalg.norm(P[:, :, 3], axis=1)
    el = np.degrees(np.arcsin(P[:, 2, 3] / r))
    assert r.min() >= 3.5 - 1e-5 and r.max() <= 4.5 + 1e-5
    assert el.min() >= -30 - 1e-4 and el.max() <= 30 + 1e-4

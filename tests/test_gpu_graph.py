"""Renders captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

sqn_render and sqn_render_stats allocate nothing, clear nothing with
memset nodes and synchronise nothing, so a serving loop can capture them
once and replay the graph for each new pose written into the captured pose
buffer.  Each case captures one render in a launch shape, then replays the
graph several times with the poses changed in between and with eager
renders of other poses interleaved, and checks every replay bit for bit
against an eager render of the same poses (the same kernel on the same
inputs).
"""
import dataclasses

import numpy as np
import pytest

from paper_2204_02585_amd import scenes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2204_02585_amd import binding  # noqa: F401  (fails loudly without libsqn.so)


def _scene(name, **kw):
    cfg = dataclasses.replace(scenes.CONFIGS[name], **kw) if kw else scenes.CONFIGS[name]
    return scenes.make_scene(cfg)


def _pose_sets(sc, n_sets):
    """The scene's poses and n_sets - 1 nearby variants (a small turn about
    the world z axis, which keeps the object in view)."""
    out = [sc.poses.astype(np.float32)]
    for k in range(1, n_sets):
        a = np.deg2rad(7.0 * k)
        rz = np.array([[np.cos(a), -np.sin(a), 0.0], [np.sin(a), np.cos(a), 0.0], [0.0, 0.0, 1.0]])
        p = sc.poses.astype(np.float64).copy()
        p[:, :, :3] = rz @ p[:, :, :3]
        p[:, :, 3] = p[:, :, 3] @ rz.T
        out.append(p.astype(np.float32))
    return out


# (workload, overrides, lanes per ray, hybrid centre fraction, views)
CASES = [
    ("tiny", {}, 0, 0.0, 1),
    ("tiny", {}, 1, 0.0, 1),
    ("tiny", {}, 4, 0.0, 1),
    ("tiny", {}, 8, 0.0, 1),
    ("tiny", {}, 0, 0.5, 1),
    ("tiny", {}, 1, 0.0, 3),
    ("paper", {"width": 96, "height": 80, "focal": 120.0}, 0, 1.0, 1),
    ("tiny_alt", {}, 4, 0.0, 1),
    ("llff_tiny", {}, 8, 0.0, 1),
]


@pytest.mark.parametrize("name,over,lanes,centre,views", CASES)
def test_graph_replays_match_eager_renders(name, over, lanes, centre, views):
    import torch
    from paper_2204_02585_amd import binding
    sc = _scene(name, **over)
    if views > 1:
        sc = scenes.make_scene(sc.config, n_poses=views)
    cfg = sc.config
    print(f"[graph {name} {cfg.width}x{cfg.height}x{views} lanes={lanes} centre={centre}]", flush=True)
    caches = binding.caches_from_scene(sc)
    caches.set_lanes_per_ray(lanes)
    if centre > 0.0:
        caches.set_centre_block(centre)
    sets = [torch.from_numpy(p).cuda() for p in _pose_sets(sc, 3)]
    args = (sc.intrinsics, sc.near, sc.far, cfg.n_samples)

    # eager references, every pose set
    refs = []
    for P in sets:
        rgb, depth, st = caches.render_stats(P, *args)
        refs.append((rgb.clone(), depth.clone(), st.clone()))
    torch.cuda.synchronize()

    # static buffers the graphs read and write
    P_static = sets[0].clone()
    B = P_static.shape[0]
    rgb_s = torch.empty((B, cfg.height, cfg.width, 3), dtype=torch.float32, device="cuda")
    depth_s = torch.empty((B, cfg.height, cfg.width), dtype=torch.float32, device="cuda")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        caches.render(P_static, *args, rgb_out=rgb_s, depth_out=depth_s)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        caches.render(P_static, *args, rgb_out=rgb_s, depth_out=depth_s)
    g_stats = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_stats):
        rgb_g, depth_g, st_g = caches.render_stats(P_static, *args)
    torch.cuda.synchronize()

    for rep, k in enumerate([1, 0, 2, 1, 2]):
        P_static.copy_(sets[k])
        rgb_s.fill_(float("nan"))
        depth_s.fill_(float("nan"))
        st_g.fill_(-1)
        g.replay()
        # eager work between replays: a render of another pose set
        other = (k + 1) % len(sets)
        e_rgb, e_depth = caches.render(sets[other], *args)
        g_stats.replay()
        torch.cuda.synchronize()
        tag = f"{name} lanes={lanes} centre={centre} replay {rep} poses {k}"
        assert torch.equal(rgb_s, refs[k][0]), tag
        assert torch.equal(depth_s, refs[k][1]), tag
        assert torch.equal(rgb_g, refs[k][0]), tag
        assert torch.equal(depth_g, refs[k][1]), tag
        assert torch.equal(st_g, refs[k][2]), tag
        assert torch.equal(e_rgb, refs[other][0]), tag
        assert torch.equal(e_depth, refs[other][1]), tag
    # the pose sets render differently, so a replay that ignored the updated
    # pose buffer would have failed above
    assert not torch.equal(refs[0][0], refs[1][0])
    del g, g_stats
    caches.close()

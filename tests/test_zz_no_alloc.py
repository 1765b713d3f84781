"""sqn_recreate_caches, the entry point for callers that cannot allocate:
new Eq. 4 caches written into an existing handle's device memory with the
create-time preparation in the library's static scratch.  Its renders must
be bit for bit those of a handle made by sqn_create_caches from the same
arrays, on two calls in a row, the second with a smaller grid."""
import ctypes
import dataclasses

import numpy as np
import pytest

from paper_2204_02585_amd import scenes

pytestmark = pytest.mark.gpu

# the first recreate: a grid of 96 nodes, binary16; the handle is created
# from another scene of the same shape (other seeds), so every array changes
BIG = scenes.Config("recreate_big", 21, 64, 48, 64, 96, 8, 32, 32, "f16", 16, 50.0, 0.1, 0.4, focal=80.0)
BIG_START = dataclasses.replace(BIG, name="recreate_start", number=22)
# the second: 48 nodes, binary32, another direction grid and D
SMALL = scenes.Config("recreate_small", 23, 40, 36, 48, 48, 4, 16, 24, "f32", 12, 50.0, 0.1, 0.4, focal=50.0)


def _device_arrays(scene):
    import torch
    sig = [torch.from_numpy(a).cuda() for a in scene.sigma]
    uvw = [torch.from_numpy(a).cuda() for a in scene.uvw]
    beta = torch.from_numpy(scene.beta).cuda()
    return sig, uvw, beta


def _desc(scene, sig, uvw, beta):
    from paper_2204_02585_amd import binding
    d = binding.CacheDesc()
    d.n_p, d.D = scene.config.n_p, scene.config.D
    d.n_theta, d.n_phi = beta.shape[0], beta.shape[1]
    d.sigma_dtype = binding._dtype_code(sig[0])
    d.uvw_dtype = binding._dtype_code(uvw[0])
    d.beta_dtype = binding._dtype_code(beta)
    d.stratified = 0
    for r in range(3):
        d.bbox_min[r], d.bbox_max[r] = scene.bbox_min[r], scene.bbox_max[r]
    d.t_eps = scene.config.t_eps
    d.reserved = 0
    d.seed = scene.seed
    return d


def _render(caches, scene):
    import torch
    P = torch.from_numpy(scene.poses).cuda()
    N = scene.config.n_samples
    rgb, depth = caches.render(P, scene.intrinsics, scene.near, scene.far, N)
    _, _, st = caches.render_stats(P, scene.intrinsics, scene.near, scene.far, N)
    torch.cuda.synchronize()
    return rgb.cpu().numpy(), depth.cpu().numpy(), st.cpu().numpy()


def _recreate(caches, scene):
    """sqn_recreate_caches through the C ABI; returns the arrays, which must
    outlive the stream's work."""
    import torch
    from paper_2204_02585_amd import binding
    sig, uvw, beta = _device_arrays(scene)
    desc = _desc(scene, sig, uvw, beta)
    sp = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in sig])
    up = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in uvw])
    stream = torch.cuda.current_stream()
    st = binding.lib.sqn_recreate_caches(caches.handle, ctypes.byref(desc), sp, up,
                                         ctypes.c_void_p(beta.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
    assert st == binding.SQN_OK, binding.last_error()
    return sig, uvw, beta


def test_recreate_matches_create_on_two_calls():
    import torch
    from paper_2204_02585_amd import binding
    start, big, small = (scenes.make_scene(c) for c in (BIG_START, BIG, SMALL))
    handle = binding.caches_from_scene(start)
    try:
        for step, scene in enumerate((big, small)):
            print(f"[recreate call {step + 1}: {scene.config.name} n_p={scene.config.n_p} "
                  f"{scene.config.dtype} D={scene.config.D}]", flush=True)
            torch.cuda.synchronize()
            free0 = torch.cuda.mem_get_info()[0]
            keep = _recreate(handle, scene)
            torch.cuda.synchronize()
            free1 = torch.cuda.mem_get_info()[0]
            if step == 1:
                # the call itself takes no device memory
                assert free1 == free0, (free0, free1)
            got = _render(handle, scene)
            del keep
            ref_caches = binding.caches_from_scene(scene)
            try:
                want = _render(ref_caches, scene)
            finally:
                ref_caches.close()
            for g, w, name in zip(got, want, ("rgb", "depth", "stats")):
                assert g.shape == w.shape, name
                assert np.array_equal(g, w), (step, name, float(np.max(np.abs(g.astype(np.float64) - w))))
            # the render is not trivially empty
            assert float(want[0].max()) > 0.05
    finally:
        handle.close()


def test_recreate_rejects_what_the_handle_cannot_hold():
    import torch
    from paper_2204_02585_amd import binding
    small, big = scenes.make_scene(SMALL), scenes.make_scene(BIG)
    handle = binding.caches_from_scene(small)
    try:
        sig, uvw, beta = _device_arrays(big)
        desc = _desc(big, sig, uvw, beta)
        sp = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in sig])
        up = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in uvw])
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        bp = ctypes.c_void_p(beta.data_ptr())
        # a layout larger than the handle's block
        st = binding.lib.sqn_recreate_caches(handle.handle, ctypes.byref(desc), sp, up, bp, stream)
        assert st == binding.SQN_ERR_INVALID_ARG and "holds" in binding.last_error()
        # a grid beyond the static scratch
        desc.n_p = 4096
        st = binding.lib.sqn_recreate_caches(handle.handle, ctypes.byref(desc), sp, up, bp, stream)
        assert st == binding.SQN_ERR_INVALID_ARG and "scratch" in binding.last_error()
        # NULL handle
        st = binding.lib.sqn_recreate_caches(None, ctypes.byref(desc), sp, up, bp, stream)
        assert st == binding.SQN_ERR_INVALID_ARG
        # the handle still renders its own caches
        got = _render(handle, small)
        ref = binding.caches_from_scene(small)
        try:
            want = _render(ref, small)
        finally:
            ref.close()
        assert all(np.array_equal(g, w) for g, w in zip(got, want))
    finally:
        handle.close()


def test_recreate_rejects_linear_handles():
    import torch
    from paper_2204_02585_amd import binding
    alt = scenes.make_scene("tiny_alt")
    plain = scenes.make_scene(SMALL)
    handle = binding.caches_from_scene(alt)
    try:
        sig, uvw, beta = _device_arrays(plain)
        desc = _desc(plain, sig, uvw, beta)
        sp = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in sig])
        up = (ctypes.c_void_p * 3)(*[t.data_ptr() for t in uvw])
        st = binding.lib.sqn_recreate_caches(handle.handle, ctypes.byref(desc), sp, up,
                                             ctypes.c_void_p(beta.data_ptr()),
                                             ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == binding.SQN_ERR_UNSUPPORTED
    finally:
        handle.close()

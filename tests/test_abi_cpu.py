"""Host-side checks of the C-ABI library that need no GPU: it loads, it
exports every function include/sqn.h declares, and argument validation that
happens before any device call returns the documented statuses."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "sqn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sqn_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2204_02585_amd import binding
    return binding


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("sqn_create_caches", "sqn_render", "sqn_destroy"):
        assert required in names


def test_library_exports_every_declared_function(lib):
    raw = ctypes.CDLL(lib.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(raw, name), name
    assert set(_declared_functions()) == set(lib.EXPORTS)


def test_status_strings(lib):
    assert lib.status_string(lib.SQN_OK) == "success"
    assert "invalid" in lib.status_string(lib.SQN_ERR_INVALID_ARG)
    assert lib.status_string(99) == "unknown status"


def test_validation_before_device_calls(lib):
    """NULL descriptors, out-of-range sizes and NULL handles are rejected by
    host code alone."""
    vp = ctypes.c_void_p
    out = vp()
    planes = (vp * 3)()
    assert lib.lib.sqn_create_caches(None, planes, planes, None, None, ctypes.byref(out)) \
        == lib.SQN_ERR_INVALID_ARG
    assert "desc" in lib.last_error()
    desc = lib.CacheDesc()
    desc.n_p, desc.D, desc.n_theta, desc.n_phi = 1, 8, 4, 4
    for r in range(3):
        desc.bbox_min[r], desc.bbox_max[r] = -1.0, 1.0
    assert lib.lib.sqn_create_caches(ctypes.byref(desc), planes, planes, None, None,
                                     ctypes.byref(out)) == lib.SQN_ERR_INVALID_ARG
    assert "n_p" in lib.last_error()
    desc.n_p = 64
    desc.D = 0
    assert lib.lib.sqn_create_caches(ctypes.byref(desc), planes, planes, None, None,
                                     ctypes.byref(out)) == lib.SQN_ERR_INVALID_ARG
    desc.D = 8
    desc.sigma_dtype = 7
    assert lib.lib.sqn_create_caches(ctypes.byref(desc), planes, planes, None, None,
                                     ctypes.byref(out)) == lib.SQN_ERR_INVALID_ARG
    desc.sigma_dtype = 0
    desc.t_eps = float("nan")
    assert lib.lib.sqn_create_caches(ctypes.byref(desc), planes, planes, None, None,
                                     ctypes.byref(out)) == lib.SQN_ERR_INVALID_ARG
    desc.t_eps = 1e-4
    desc.n_p, desc.D = 8192, 32
    assert lib.lib.sqn_create_caches(ctypes.byref(desc), planes, planes, None, None,
                                     ctypes.byref(out)) == lib.SQN_ERR_UNSUPPORTED
    # a direction cache the 32-bit offsets cannot address (2^31 binary32 values)
    desc.n_p, desc.D = 64, 8
    desc.n_theta, desc.n_phi = 65536, 4096
    assert lib.lib.sqn_create_caches(ctypes.byref(desc), planes, planes, None, None,
                                     ctypes.byref(out)) == lib.SQN_ERR_UNSUPPORTED
    assert "direction cache" in lib.last_error()
    desc.n_theta, desc.n_phi = 4, 4
    intr = lib.Intrinsics(1.0, 1.0, 0.5, 0.5, 1, 1)
    assert lib.lib.sqn_render(None, None, 1, ctypes.byref(intr), 2.0, 6.0, 8, None, None,
                              None) == lib.SQN_ERR_INVALID_ARG
    assert lib.lib.sqn_cache_device_bytes(None) == 0
    lib.lib.sqn_destroy(None)


def test_linear_decoder_validation_before_device_calls(lib):
    """sqn_create_linear_caches rejects a NULL decoder, d_sigma outside
    [1, 64], NULL weight arrays and non-finite weights before touching the
    device."""
    import numpy as np
    vp = ctypes.c_void_p
    out = vp()
    planes = (vp * 3)()
    desc = lib.CacheDesc()
    desc.n_p, desc.D, desc.n_theta, desc.n_phi = 64, 2, 4, 4
    for r in range(3):
        desc.bbox_min[r], desc.bbox_max[r] = -1.0, 1.0
    desc.t_eps = 1e-4
    ws = np.ones(3 * 4, np.float32)
    wu = np.ones((3, 2, 6), np.float32)
    bu = np.zeros((3, 2), np.float32)

    def create(dec):
        return lib.lib.sqn_create_linear_caches(ctypes.byref(desc), dec, planes, planes, None,
                                                None, ctypes.byref(out))

    def dec(ds=4, b=0.0, w_s=ws, w_u=wu, b_u=bu):
        return ctypes.byref(lib.LinearDecoder(ds, b, w_s.ctypes.data if w_s is not None else None,
                                              w_u.ctypes.data if w_u is not None else None,
                                              b_u.ctypes.data if b_u is not None else None))

    assert create(None) == lib.SQN_ERR_INVALID_ARG and "decoder" in lib.last_error()
    assert create(dec(ds=0)) == lib.SQN_ERR_INVALID_ARG and "d_sigma" in lib.last_error()
    assert create(dec(ds=65)) == lib.SQN_ERR_INVALID_ARG
    assert create(dec(w_s=None)) == lib.SQN_ERR_INVALID_ARG
    assert create(dec(b=float("inf"))) == lib.SQN_ERR_INVALID_ARG
    wu[2, 1, 5] = np.nan
    assert create(dec()) == lib.SQN_ERR_INVALID_ARG and "w_uvw[35]" in lib.last_error()
    wu[2, 1, 5] = 1.0
    # a valid decoder reaches the plane checks
    assert create(dec()) == lib.SQN_ERR_INVALID_ARG and "sigma_planes" in lib.last_error()
    assert not out


def test_probe_library_exports_and_rejects_bad_sizes():
    """The benchmark's ceiling probes (libsqn_probe.so: memory levels, the
    vector-memory data path and matrix cores) load and reject sizes they
    cannot measure before touching the device."""
    from paper_2204_02585_amd import build
    raw = ctypes.CDLL(build.PROBE_PATH)
    raw.sqn_probe_stream.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    raw.sqn_probe_gather.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(ctypes.c_float)]
    ms = ctypes.c_float()
    assert raw.sqn_probe_stream(15, 1, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_stream(1 << 20, 0, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_stream(1 << 20, 1, None) == 1
    raw.sqn_probe_stream_nt.argtypes = raw.sqn_probe_stream.argtypes
    assert raw.sqn_probe_stream_nt(15, 1, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_stream_nt(1 << 20, 0, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_gather(100, 1, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_gather(1 << 20, 0, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_gather(64 << 32, 1, ctypes.byref(ms)) == 1
    raw.sqn_probe_mfma_f16.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    assert raw.sqn_probe_mfma_f16(0, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_mfma_f16(10, None) == 1
    raw.sqn_probe_vmem.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                   ctypes.POINTER(ctypes.c_float)]
    assert raw.sqn_probe_vmem(2, 0, 16, 2.4, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_vmem(0, 2, 16, 2.4, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_vmem(0, 0, 0, 2.4, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_vmem(0, 0, 16, 0.0, ctypes.byref(ms)) == 1
    assert raw.sqn_probe_vmem(0, 0, 16, 2.4, None) == 1

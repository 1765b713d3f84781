#!/usr/bin/env python3
"""Throughput of the cached SqueezeNeRF render path on one MI355X.

One step = one sqn_render call over one batch of views (the whole hot path:
ray generation, sample placement, cache gathers, beta . uvw colour and
compositing).  Inputs (caches, poses, output buffers) are resident in HBM
before the timed region.  Prints ONE JSON line.

Default workload: 800x800 pixels, 192 samples per ray, position sub-caches
k=256 with D=8 in fp16, 128x128 fp16 direction cache, 64 seeded blobs.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Msamples/s and frames/s at 800x800x192 samples; achieved GB/s vs HBM peak"
HBM_PEAK_GBS = 8000.0

WORKLOAD_TEXT = {
    "tiny": "64x64 image, 64 uniform samples/ray, k=64 D=8 fp32 caches, 32x32 fp32 direction cache, 16 blobs",
    "paper": "800x800 image, 192 uniform samples/ray, k=256 D=8 fp16 caches, 128x128 fp16 direction cache, 64 blobs sigma_max 50",
    "paper512": "800x800 image, 256 uniform samples/ray, the paper's 512 cache (k=512, sigma fp32, uvw fp16, D=8), 64x64 fp16 direction cache, 64 blobs sigma_max 50",
    "large": "800x800 image, 192 uniform samples/ray, k=1024 D=8 fp16 caches, 384x384 fp16 direction cache, 64 blobs sigma_max 200",
    "batch": "100 spiral views of 800x800, 192 uniform samples/ray, k=256 D=8 fp16 caches, 128x128 fp16 direction cache",
    "stress": "1920x1080 image, 384 stratified samples/ray, k=2048 D=16 fp16 caches, 512x512 fp16 direction cache, 256 blobs",
    "llff": "forward-facing (LLFF-shaped), rays in NDC: 504x378 image, 256 uniform samples/ray, the paper's 512 cache (sigma fp32, uvw fp16, D=8), 32x32 fp16 direction cache, 64 blobs in the NDC box",
    "alt": "Eq. 5 linear decoder (D_sigma=12): 800x800 image, 192 uniform samples/ray, k=256 D=8 fp16 caches, 128x128 fp16 direction cache, 64 blobs",
    "alt512": "Eq. 5 linear decoder (D_sigma=12) at the paper's alt cache size: 800x800 image, 192 uniform samples/ray, k=512 D=8 fp16 caches, 256x256 fp16 direction cache, 64 blobs",
}


def algorithmic_bytes(cfg, n_rays, live_inbox, occupied):
    """Bytes the method must move per launch: per ray the 4 direction-cache
    texels (D values each), the pose row reads are broadcast and not
    counted, 16 B of output (rgb + depth); per live in-box sample the three
    sigma^j (for the Eq. 5 decoder the three binary32 per-plane partial
    sums the caches are folded into; its radiance weights are read once per
    ray from cache and not counted); per live occupied sample the three uvw
    records (3D values)."""
    b = 2 if cfg.dtype == "f16" else 4
    b_sigma = 4 if (cfg.sigma_channels > 0 or (cfg.sigma_dtype or cfg.dtype) == "f32") else 2
    per_ray = 4 * cfg.D * b + 16
    return n_rays * per_ray + live_inbox * 3 * b_sigma + occupied * 3 * 3 * cfg.D * b


# Cycles per second of the vector-memory data path (TD) over all CUs:
# 256 CUs x 2.4 GHz.  Access-pattern probes on this GPU keep TD busy on every
# cycle, and each gather's busy cycles match its cost there.
TD_PEAK_GCYCLES = 256 * 2.4
CLOCK_GHZ = 2.4


def counter_record(config_name, kind="render", lanes=None):
    """The committed rocprofv3 counter record of a workload's kernel
    (profiles/<kind>_traffic_<workload>.json): HBM bytes per launch from the
    FETCH_SIZE / WRITE_SIZE passes scaled by kernels of known traffic, and
    for render kernels the TD busy cycles, L1 accesses and VALU
    instructions per launch.  None when no such file exists, the kernel
    source has changed since the counters were taken, or (lanes given) the
    record is of a kernel with another number of lanes per ray."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kind}_traffic_{config_name}.json")
    src = os.path.join(ROOT, "paper_2204_02585_amd", "csrc", f"{kind}.hip")
    try:
        rec = json.load(open(path))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    except (OSError, ValueError):
        return None
    if rec.get(f"{kind}_hip_sha256_16") != sha:
        return None
    if lanes and (f"L={lanes}," if lanes > 0 else "hybrid") not in rec.get("kernel", ""):
        return None
    return rec


def measured_traffic(config_name, kind="render"):
    rec = counter_record(config_name, kind)
    return None if rec is None else int(rec["traffic_bytes_per_launch"])


def render_roofline(rec, ms, bytes_alg):
    """Roofline of the render kernel against the unit its counters show
    busiest, the vector-memory data path (TD): achieved = TD busy CU-cycles
    per launch (committed counters of this kernel) over the launch time
    measured here, so frac is the fraction of the launch the data path is
    busy.  VALU issue per CU per clock from the same counters; the method's
    algorithmic bytes per launch (sigma^j of every live in-box sample, three
    uvw records per occupied one, beta corners and outputs per ray) as the
    rate the kernel serves them; HBM bytes from the FETCH/WRITE counters
    against the 8 TB/s HBM peak."""
    sec = ms * 1e-3
    td = None if rec is None else rec.get("td_busy_cycles_per_launch")
    achieved = None if td is None else td / sec / 1e9
    traffic = None if rec is None else int(rec["traffic_bytes_per_launch"])
    valu = None if rec is None else rec.get("valu_insts_per_launch")
    return {"bound": "vmem", "achieved": None if achieved is None else round(achieved, 2),
            "peak": round(TD_PEAK_GCYCLES, 1), "unit": "G busy cycles/s of the TD data path, all CUs",
            "frac": None if achieved is None else round(achieved / TD_PEAK_GCYCLES, 4),
            "traffic": traffic,
            "basis": "rocprofv3 TD_TD_BUSY_sum of this kernel per launch (profiles/) / launch time measured "
                     "here; peak = 256 CUs x 2.4 GHz",
            "td_busy_cycles_per_launch": None if td is None else int(td),
            "valu_insts_per_cu_clock": None if valu is None else round(valu / (256 * CLOCK_GHZ * 1e9 * sec), 3),
            "served_algorithmic_gbs": round(bytes_alg / sec / 1e9, 1),
            "algorithmic_bytes_per_launch": int(bytes_alg),
            "hbm_gbs": None if traffic is None else round(traffic / sec / 1e9, 1),
            "hbm_frac": None if traffic is None else round(traffic / sec / 1e9 / HBM_PEAK_GBS, 4),
            "kernel_ms_per_launch": round(ms, 5)}


# Launch shape per workload (lanes per ray, hybrid centre fraction): the
# fastest that sqn_tune_lanes_per_ray measured for it on one MI355X (the
# candidates' times are within a few percent of run-to-run spread where two
# are close, so the bench fixes the shape its committed counters describe;
# --tune measures again).
LAUNCH_SHAPES = {"paper": (1, 0.0), "large": (0, 1.0), "paper512": (0, 1.0), "stress": (1, 0.0),
                 "batch": (1, 0.0), "alt": (4, 0.0), "alt512": (4, 0.0), "llff": (8, 0.0), "tiny": (8, 0.0)}

# Worker threads a process on a one-GPU share of the shared host may use.
HOST_CPU_SHARE = 16


def host_description():
    """The host the CPU baseline runs on: logical CPUs, the CPUs this
    process may run on, physical cores and the CPU model (/proc/cpuinfo)."""
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = os.cpu_count() or 1
    model, cores = None, set()
    try:
        phys = core = None
        with open("/proc/cpuinfo") as f:
            for line in f:
                key, _, val = line.partition(":")
                key, val = key.strip(), val.strip()
                if key == "model name" and model is None:
                    model = val
                elif key == "physical id":
                    phys = val
                elif key == "core id":
                    core = val
                elif not key and phys is not None and core is not None:
                    cores.add((phys, core))
                    phys = core = None
        if phys is not None and core is not None:
            cores.add((phys, core))
    except OSError:
        pass
    return {"host_logical_cpus": os.cpu_count(), "affinity_cpus": affinity,
            "host_physical_cores": len(cores) or None, "cpu_model": model}


def baseline_threads():
    """All CPUs this process may run on, up to the CPU share of one GPU."""
    return max(1, min(HOST_CPU_SHARE, host_description()["affinity_cpus"]))


def cpu_baseline(scene, budget_s=12.0, max_frames=40):
    """The CPU oracle as it stands, on whole frames of the same workload,
    repeated until ~budget_s of wall time (at least one frame): view 0 of a
    single view, every 10th view of a batch in turn (views differ in cost).
    Threads: every CPU the process may use, capped at the host's CPU share
    for one GPU (HOST_CPU_SHARE)."""
    import oracle
    host = host_description()
    threads = baseline_threads()
    cfg = scene.config
    views = list(range(0, scene.poses.shape[0], 10))
    frames = 0
    t0 = time.perf_counter()
    while True:
        v = views[frames % len(views)]
        oracle.render_scene(scene, poses=scene.poses[v:v + 1], n_threads=threads)
        frames += 1
        el = time.perf_counter() - t0
        if el >= budget_s or frames >= max_frames:
            break
    samples = frames * cfg.width * cfg.height * cfg.n_samples
    which = "view 0" if len(views) == 1 else f"views {', '.join(map(str, views))} in turn"
    return {"value": samples / el / 1e6, "unit": "Msamples/s", "cores": threads, "kind": "oracle",
            "sample": f"{frames} full {cfg.width}x{cfg.height}x{cfg.n_samples} frame(s) of {which}, "
                      f"{el:.1f} s wall", "frames_per_s": frames / el,
            "threads": threads, "thread_cap": HOST_CPU_SHARE, **host}


def memory_ceilings(cache_bytes):
    """Ceilings of the memory levels the render kernel's gathers are served
    from, measured on this GPU by libsqn_probe.so: streaming reads of a
    2 MiB buffer (held by each XCD's L2), a 128 MiB buffer (held by the
    MALL) and a 4 GiB buffer (HBM; also with non-temporal loads, the
    streaming ceiling of HBM), and random 64-byte-record gathers over
    buffers of those sizes and of the workload's cache size.  GB/s."""
    import ctypes
    from paper_2204_02585_amd import build as _build
    lib = ctypes.CDLL(_build.PROBE_PATH)
    lib.sqn_probe_stream.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    lib.sqn_probe_stream_nt.argtypes = lib.sqn_probe_stream.argtypes
    lib.sqn_probe_gather.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(ctypes.c_float)]
    ms = ctypes.c_float()
    out = {"stream_gbs": {}, "gather64_gbs": {}}
    for label, nbytes, passes, probe in (("2MiB", 2 << 20, 2000, lib.sqn_probe_stream),
                                         ("128MiB", 128 << 20, 16, lib.sqn_probe_stream),
                                         ("4GiB", 4 << 30, 1, lib.sqn_probe_stream),
                                         ("4GiB_nontemporal", 4 << 30, 1, lib.sqn_probe_stream_nt)):
        if probe(nbytes, passes, ctypes.byref(ms)) != 0:
            raise RuntimeError("stream probe failed")
        out["stream_gbs"][label] = round(nbytes * passes / (ms.value * 1e-3) / 1e9, 1)
    cache_label = f"cache {cache_bytes / 1e6:.1f} MB"
    n_rec = 1 << 24
    for label, nbytes in (("2MiB", 2 << 20), (cache_label, (int(cache_bytes) + 63) // 64 * 64),
                          ("128MiB", 128 << 20), ("4GiB", 4 << 30)):
        if lib.sqn_probe_gather(nbytes, n_rec, ctypes.byref(ms)) != 0:
            raise RuntimeError("gather probe failed")
        out["gather64_gbs"][label] = round(n_rec * 64 / (ms.value * 1e-3) / 1e9, 1)
    out["cache_label"] = cache_label
    return out


# lane patterns of the render kernel's loads: the sigma gathers are dword
# loads with every lane in its own 64-byte segment (a quad holds four
# samples of one ray, texels apart), the colour records 16-byte loads
VMEM_PATTERNS = (("dword_lane_per_segment", 0, 0), ("dword_quad_per_segment", 0, 1),
                 ("dwordx4_lane_per_segment", 1, 0), ("dwordx4_quad_per_segment", 1, 1))


def vmem_ceiling():
    """Cycles per wave-level load instruction on one CU with the
    vector-memory data path saturated by gathers that the vector L1 serves
    (libsqn_probe.so), for dword and 16-byte loads with every lane in its own
    64-byte segment or a quad sharing one: what a load costs the path that
    the render kernel's TD-busy fraction measures."""
    import ctypes
    from paper_2204_02585_amd import build as _build
    lib = ctypes.CDLL(_build.PROBE_PATH)
    lib.sqn_probe_vmem.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                   ctypes.POINTER(ctypes.c_float)]
    cyc = ctypes.c_float()
    out = {}
    for label, wide, quads in VMEM_PATTERNS:
        if lib.sqn_probe_vmem(wide, quads, 256, CLOCK_GHZ, ctypes.byref(cyc)) != 0:
            raise RuntimeError("vector-memory probe failed")
        out[label] = round(cyc.value, 2)
    return out


def mfma_ceiling():
    """Dense binary16 matrix-core rate of this GPU at two waves per SIMD
    (independent 32x32x16 products, libsqn_probe.so), TFLOP/s."""
    import ctypes
    from paper_2204_02585_amd import build as _build
    lib = ctypes.CDLL(_build.PROBE_PATH)
    lib.sqn_probe_mfma_f16.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    tf = ctypes.c_float()
    if lib.sqn_probe_mfma_f16(2000, ctypes.byref(tf)) != 0:
        raise RuntimeError("matrix-core probe failed")
    return round(tf.value, 1)


def calibration_copies(dev):
    """Kernels of known traffic for scaling the hardware byte counters: a
    1 GiB fill and three 1 GiB device-to-device copies."""
    import torch
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


GEN_TEXT = {
    "gen_tiny": "cache generation: 3 position networks (6x256) on 32x32 grids, direction network (4x128) on 16x16 nodes, D=8",
    "gen_512": "cache generation for the paper's 512 cache: 3 position networks (6x256, NeRF encoding L=10) on 512x512 grids, direction network (4x128, L=4) on 64x64 nodes, D=8",
    "gen_1k": "cache generation for the paper's 1K cache (Table 4): 3 position networks (6x256, NeRF encoding L=10) on 1024x1024 grids, direction network (4x128, L=4) on 64x64 nodes, D=8",
}
MFMA_F16_PEAK_TFLOPS = 2500.0


def network_flops(cfg):
    """Multiply-adds x 2 of the networks as specified (unpadded): per
    position point n_in W + (L - 1) W^2 + W n_out, per direction node the
    same with the direction shapes."""
    pos = cfg.pos_in * cfg.pos_width + (cfg.pos_layers - 1) * cfg.pos_width ** 2 + cfg.pos_width * cfg.pos_out
    dirn = cfg.dir_in * cfg.dir_width + (cfg.dir_layers - 1) * cfg.dir_width ** 2 + cfg.dir_width * cfg.D
    return 2 * pos, 2 * dirn


def bench_generate(args):
    """One step = one sqn_generate_caches call: all three position grids and
    the direction grid, written into resident output buffers."""
    import torch
    from paper_2204_02585_amd import binding, scenes
    g = scenes.make_gen_scene(args.config)
    cfg = g.config
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    nets = binding.networks_from_gen_scene(g)
    n_pos = 3 * cfg.n_p * cfg.n_p
    n_dir = cfg.n_theta * cfg.n_phi
    out = ([torch.empty((cfg.n_p, cfg.n_p), dtype=torch.float32, device=dev) for _ in range(3)],
           [torch.empty((cfg.n_p, cfg.n_p, 3 * cfg.D), dtype=torch.float16, device=dev) for _ in range(3)],
           torch.empty((cfg.n_theta, cfg.n_phi, cfg.D), dtype=torch.float16, device=dev))
    stream = torch.cuda.current_stream()

    def step():
        nets.generate(cfg.n_p, cfg.n_theta, cfg.n_phi, g.bbox_min, g.bbox_max, out=out, stream=stream)

    # untimed settle of the GPU clocks (as for the render workloads), then
    # the warm-up steps
    print(f"[bench] {cfg.name}: settle {args.settle} s, warmup {args.warmup}", file=sys.stderr, flush=True)
    settle0 = time.perf_counter()
    settle_calls = 0
    while time.perf_counter() - settle0 < args.settle:
        step()
        settle_calls += 1
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = ev0.elapsed_time(ev1) / args.steps
    f_pos, f_dir = network_flops(cfg)
    flops = n_pos * f_pos + n_dir * f_dir
    tflops = flops / (ms * 1e-3) / 1e12
    if args.copy_calibration:
        calibration_copies(dev)

    base = None
    if not args.no_cpu_baseline:
        # the binary64 oracle on a bounded sample of position points
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        import numpy as np
        from oracle import cachegen
        rng = np.random.Generator(np.random.PCG64(1))
        n_s = 0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_budget and n_s < 3 * 65536:
            ia = rng.integers(0, cfg.n_p, 8192)
            ib = rng.integers(0, cfg.n_p, 8192)
            cachegen.position_cache_points(g.pos[n_s % 3], cfg.n_p, n_s % 3, g.bbox_min, g.bbox_max, cfg.D,
                                           ia, ib, cfg.pos_freq)
            n_s += 8192
        el = time.perf_counter() - t0
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 1)
        base = {"value": round(n_s / el / 1e6, 4), "unit": "Mpoints/s", "cores": threads, "kind": "oracle",
                "sample": f"{n_s} random position-grid points (binary64 numpy, BLAS threads as configured), "
                          f"{el:.1f} s wall", "threads": threads, **host_description()}
    nets.close()
    ceilings = None
    if not args.no_ceilings:
        print("[bench] matrix-core ceiling", file=sys.stderr, flush=True)
        peak = mfma_ceiling()
        ceilings = {"mfma_f16_tflops": peak, "kernel_vs_mfma_ceiling": round(tflops / peak, 4)}
    out_line = {
        "metric": "cache generation: Mpoints/s of network evaluations on the cache grids",
        "value": round((n_pos + n_dir) / (ms * 1e-3) / 1e6, 2),
        "unit": "Mpoints/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": {"seconds": args.settle, "calls": settle_calls},
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded He-uniform binary16 weights; no trained networks)",
        "config": {"workload": f"{cfg.name}: {GEN_TEXT[cfg.name]}", "n_p": cfg.n_p,
                   "direction_grid": [cfg.n_theta, cfg.n_phi], "D": cfg.D,
                   "position_points": n_pos, "direction_points": n_dir},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_F16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / MFMA_F16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(cfg.name, "generate"),
                     "algorithmic_flops_per_launch": int(flops), "kernel_ms_per_launch": round(ms, 4)},
        "cpu_baseline": base,
        "ceilings": ceilings,
        "wall_s_timed": round(wall, 4),
    }
    print(json.dumps(out_line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="paper", choices=sorted(WORKLOAD_TEXT) + sorted(GEN_TEXT),
                    help="a render workload, or gen_* for cache generation")
    ap.add_argument("--lanes", type=int, default=0,
                    help="lanes of a wavefront per ray (1, 4 or 8); 0 with --centre 0 = the workload's "
                         "recorded launch shape")
    ap.add_argument("--dense", action="store_true",
                    help="march every sample (no leaps over empty space)")
    ap.add_argument("--centre", type=float, default=0.0,
                    help="hybrid launch of a single view: centred fraction of 16-pixel blocks with four lanes per "
                         "ray (sqn_set_centre_block); 0 = off")
    ap.add_argument("--settle", type=float, default=0.1,
                    help="seconds of untimed rendering before the warm-up steps (the GPU clocks settle)")
    ap.add_argument("--tune", action="store_true",
                    help="time the launch shapes with sqn_tune_lanes_per_ray instead of the workload's recorded one")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the ceiling probes (memory levels; matrix cores for gen_*)")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--vmem-probe", action="store_true",
                    help="only run the vector-memory saturation probe and print its cycles per load")
    ap.add_argument("--graph", type=int, default=0,
                    help="also time a serving loop that replays a HIP graph of this many captured renders "
                         "(reported as graph_replay, beside the eager figures; 0 = off)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy 1 GiB device-to-device 3 times (a kernel "
                         "of known traffic for scaling hardware byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the render path has no cross-GPU step; "
              "run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.vmem_probe:
        print(json.dumps({"vmem_cycles_per_wave_load": vmem_ceiling(), "clock_ghz": CLOCK_GHZ}), flush=True)
        return

    if args.config in GEN_TEXT:
        bench_generate(args)
        return

    import torch
    from paper_2204_02585_amd import binding, scenes

    print(f"[bench] config={args.config} building scene", file=sys.stderr, flush=True)
    scene = scenes.make_scene(args.config)
    cfg = scene.config
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    caches = binding.caches_from_scene(scene, device=dev)
    caches.set_lanes_per_ray(args.lanes)
    caches.set_empty_space_skipping(not args.dense)
    poses = torch.from_numpy(scene.poses).to(dev)
    B = poses.shape[0]
    rgb = torch.empty((B, cfg.height, cfg.width, 3), dtype=torch.float32, device=dev)
    depth = torch.empty((B, cfg.height, cfg.width), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    N = cfg.n_samples
    lanes, centre = args.lanes, args.centre
    if args.tune:
        # the library times its launch shapes on this batch and keeps the
        # fastest (outside the timed region, like any warm-up)
        print("[bench] tuning the launch shape", file=sys.stderr, flush=True)
        lanes = caches.tune_lanes_per_ray(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth,
                                          stream=stream)
        centre = caches.centre_block
        shape_label = f"tuned: hybrid {centre:g}" if lanes == -1 else f"tuned: {lanes}"
    else:
        if lanes == 0 and centre == 0.0 and not args.dense:
            lanes, centre = LAUNCH_SHAPES.get(cfg.name, (0, 0.0))
        if centre > 0.0:
            caches.set_lanes_per_ray(0)
            caches.set_centre_block(centre)
            lanes = -1
        else:
            caches.set_lanes_per_ray(lanes)
        shape_label = f"hybrid {centre:g}" if lanes == -1 else (lanes or "auto")

    # untimed diagnostics pass: live / occupied sample counts for the byte model
    _, _, st = caches.render_stats(poses, scene.intrinsics, scene.near, scene.far, N)
    torch.cuda.synchronize()
    st = st.cpu().numpy().view(np.uint32).reshape(-1, 4)
    live_inbox = int(st[:, 1].astype(np.int64).sum())
    occupied = int(st[:, 2].astype(np.int64).sum())
    n_rays = B * cfg.width * cfg.height
    bytes_alg = algorithmic_bytes(cfg, n_rays, live_inbox, occupied)

    # the GPU's clocks take tens of milliseconds of load to settle after the
    # process starts (the same launch runs up to 8% slower at first): render
    # for args.settle seconds, untimed, before the warm-up steps
    print(f"[bench] settle {args.settle} s, warmup {args.warmup}", file=sys.stderr, flush=True)
    settle0 = time.perf_counter()
    settle_calls = 0
    while time.perf_counter() - settle0 < args.settle:
        for _ in range(4):
            caches.render(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth, stream=stream)
        settle_calls += 4
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        caches.render(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth, stream=stream)
    torch.cuda.synchronize()

    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        caches.render(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth, stream=stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = ev0.elapsed_time(ev1) / args.steps

    # spread over launches: the same launches again, each between two events
    # (outside the timed region)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for i in range(args.steps):
        caches.render(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth, stream=stream)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    spread = {"median": round(per[len(per) // 2], 5), "min": round(per[0], 5), "max": round(per[-1], 5)}

    graph_replay = None
    if args.graph > 0:
        graph_replay = time_graph_replay(caches, poses, scene, N, rgb, depth, args.graph, args.steps, ms)

    nominal = cfg.nominal_samples
    msps = nominal / (ms * 1e-3) / 1e6
    fps = B / (ms * 1e-3)
    gbs = bytes_alg / (ms * 1e-3) / 1e9

    if args.copy_calibration:
        calibration_copies(dev)
    ceilings = None
    if not args.no_ceilings:
        print("[bench] memory ceilings", file=sys.stderr, flush=True)
        ceilings = memory_ceilings(scene.cache_nbytes())
        g = ceilings["gather64_gbs"][ceilings.pop("cache_label")]
        ceilings["render_vs_gather64_at_cache_size"] = round(gbs / g, 4)
        ceilings["vmem_cycles_per_wave_load"] = vmem_ceiling()

    base = None
    if not args.no_cpu_baseline:
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        base = cpu_baseline(scene, budget_s=args.cpu_budget)
    caches.close()

    out = {
        "metric": METRIC,
        "value": round(msps, 2),
        "unit": "Msamples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": {"seconds": args.settle, "renders": settle_calls},
        "ms_per_step": round(ms, 5),
        "ms_per_launch": spread,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded blob density, uniform uvw and beta; no trained caches)",
        "config": {"workload": f"{cfg.name}: {WORKLOAD_TEXT[cfg.name]}",
                   "views_per_step": B, "width": cfg.width, "height": cfg.height,
                   "samples_per_ray": N, "n_p": cfg.n_p, "D": cfg.D, "cache_dtype": cfg.dtype,
                   "direction_cache": [cfg.n_theta, cfg.n_phi], "t_eps": cfg.t_eps,
                   "decoder": ("Eq. 5 linear, D_sigma=%d" % cfg.sigma_channels
                               if cfg.sigma_channels > 0 else "Eq. 4 product/sum"),
                   "lanes_per_ray": shape_label,
                   "empty_space_leaps": not args.dense},
        "frames_per_s": round(fps, 2),
        "samples": {"nominal_per_step": nominal, "live_inbox_per_step": live_inbox,
                    "occupied_per_step": occupied,
                    "empty_fraction_of_live_inbox": round(1.0 - occupied / live_inbox, 4) if live_inbox else None,
                    "live_inbox_msamples_per_s": round(live_inbox / (ms * 1e-3) / 1e6, 1),
                    "occupied_msamples_per_s": round(occupied / (ms * 1e-3) / 1e6, 1)},
        "roofline": render_roofline(counter_record(cfg.name, lanes=lanes) if lanes != 0 and not args.dense
                                    else None, ms, bytes_alg),
        "cpu_baseline": base,
        "ceilings": ceilings,
        "wall_s_timed": round(wall, 4),
    }
    if graph_replay is not None:
        out["graph_replay"] = graph_replay
    print(json.dumps(out), flush=True)


def time_graph_replay(caches, poses, scene, N, rgb, depth, per_graph, steps, eager_ms):
    """A serving loop's launch pattern: `per_graph` renders captured once in
    a HIP graph (torch.cuda.CUDAGraph; the renders allocate nothing and
    issue no memset), the graph replayed until about `steps` renders ran,
    between two HIP events.  Outside the timed region of `value`."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        caches.render(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(per_graph):
            caches.render(poses, scene.intrinsics, scene.near, scene.far, N, rgb, depth)
    reps = max(1, steps // per_graph)
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(reps):
        g.replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / (reps * per_graph)
    del g
    return {"renders_per_graph": per_graph, "renders_timed": reps * per_graph,
            "ms_per_render": round(ms, 5), "eager_ms_per_render": round(eager_ms, 5),
            "eager_over_graph": round(eager_ms / ms, 3)}


if __name__ == "__main__":
    main()

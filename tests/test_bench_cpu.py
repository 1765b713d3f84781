"""Host logic of bench.py (no GPU): the roofline arithmetic, the committed
counter records against the current kernel sources, the single-GPU guard and
the byte model of the method."""
import hashlib
import json
import os
import subprocess
import sys

import pytest

import bench
from paper_2204_02585_amd import scenes

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RENDER_WORKLOADS = ["tiny", "paper", "large", "batch", "stress", "alt", "alt512", "llff", "paper512"]


def test_launch_shapes_cover_every_render_workload():
    assert set(bench.LAUNCH_SHAPES) == set(RENDER_WORKLOADS)
    assert set(RENDER_WORKLOADS) <= set(bench.WORKLOAD_TEXT)
    for lanes, centre in bench.LAUNCH_SHAPES.values():
        assert lanes in (0, 1, 4, 8) and 0.0 <= centre <= 1.0
        # a hybrid launch leaves the lanes to the library, a fixed lane
        # count has no centre block
        assert (lanes == 0) == (centre > 0.0)


@pytest.mark.parametrize("name", RENDER_WORKLOADS)
def test_committed_counters_describe_the_current_kernel(name):
    """The bench line's roofline reads profiles/render_traffic_<name>.json; it
    must be of the current render.hip and of the launch shape the bench
    times, or the roofline fraction would come out null."""
    lanes, centre = bench.LAUNCH_SHAPES[name]
    rec = bench.counter_record(name, lanes=-1 if centre > 0.0 else lanes)
    src = open(os.path.join(ROOT, "paper_2204_02585_amd", "csrc", "render.hip"), "rb").read()
    raw = json.load(open(os.path.join(ROOT, "profiles", f"render_traffic_{name}.json")))
    assert raw["render_hip_sha256_16"] == hashlib.sha256(src).hexdigest()[:16], \
        f"profiles/render_traffic_{name}.json was taken on another render.hip"
    assert rec is not None, f"counter record of {name} does not match its launch shape {lanes, centre}"
    assert rec["workload"] == name
    for key in ("traffic_bytes_per_launch", "td_busy_cycles_per_launch", "valu_insts_per_launch",
                "kernel_us_trace"):
        assert rec[key] > 0
    # the data path cannot be busy for more cycles than the launch has
    assert rec["td_busy_cycles_per_launch"] <= 256 * 2.4e3 * rec["kernel_us_trace"]


def test_counter_record_rejects_other_shapes_and_missing_files():
    assert bench.counter_record("no_such_workload") is None
    # large's record is of the hybrid launch, paper's of the one-lane kernel
    assert bench.counter_record("large", lanes=1) is None
    assert bench.counter_record("large", lanes=-1) is not None
    assert bench.counter_record("paper", lanes=-1) is None
    assert bench.counter_record("paper", lanes=1) is not None
    # alt's record is of the four-lane kernel
    assert bench.counter_record("alt", lanes=8) is None
    assert bench.counter_record("alt", lanes=4) is not None


def test_render_roofline_is_a_fraction_of_the_data_path():
    rec = {"td_busy_cycles_per_launch": 55_000_000, "traffic_bytes_per_launch": 42_000_000,
           "valu_insts_per_launch": 68_000_000}
    ms = 0.1
    r = bench.render_roofline(rec, ms, bytes_alg=1.1e9)
    assert r["bound"] == "vmem"
    assert r["peak"] == pytest.approx(614.4)
    # 55e6 busy CU-cycles in 0.1 ms over 256 CUs x 2.4 GHz
    assert r["frac"] == pytest.approx(55e6 / (256 * 2.4e9 * 1e-4), abs=1e-4)
    assert 0.0 < r["frac"] <= 1.0
    assert r["achieved"] == pytest.approx(r["frac"] * r["peak"], rel=1e-3)
    assert r["traffic"] == 42_000_000
    assert r["hbm_gbs"] == pytest.approx(420.0)
    assert r["hbm_frac"] == pytest.approx(420.0 / 8000.0, abs=1e-4)
    assert r["served_algorithmic_gbs"] == pytest.approx(11000.0)
    empty = bench.render_roofline(None, ms, bytes_alg=1.1e9)
    assert empty["frac"] is None and empty["traffic"] is None and empty["achieved"] is None


def test_algorithmic_bytes_follow_the_method():
    """Per ray: four direction-cache texels of D values and 16 bytes of
    output; per live in-box sample three sigma^j; per occupied sample three
    records of 3D values."""
    paper = scenes.CONFIGS["paper"]            # fp16 everywhere, D = 8
    assert bench.algorithmic_bytes(paper, 1, 0, 0) == 4 * 8 * 2 + 16
    assert bench.algorithmic_bytes(paper, 0, 1, 0) == 3 * 2
    assert bench.algorithmic_bytes(paper, 0, 0, 1) == 3 * 3 * 8 * 2
    tiny = scenes.CONFIGS["tiny"]              # fp32 everywhere
    assert bench.algorithmic_bytes(tiny, 0, 1, 1) == 3 * 4 + 3 * 3 * 8 * 4
    p512 = scenes.CONFIGS["paper512"]          # sigma fp32, uvw fp16
    assert bench.algorithmic_bytes(p512, 0, 1, 1) == 3 * 4 + 3 * 3 * 8 * 2
    stress = scenes.CONFIGS["stress"]          # D = 16: 96-byte records
    assert bench.algorithmic_bytes(stress, 0, 0, 1) == 3 * 96
    alt = scenes.CONFIGS["alt"]                # Eq. 5: binary32 partial sums
    assert bench.algorithmic_bytes(alt, 0, 1, 0) == 3 * 4
    # the dense bound of the paper view, every sample live and occupied: the
    # survey's 150 B per sample at 800x800x192, 18.4 GB per frame
    n = paper.width * paper.height
    dense = bench.algorithmic_bytes(paper, n, n * paper.n_samples, n * paper.n_samples)
    assert dense / (n * paper.n_samples) == pytest.approx(150.0, abs=0.5)
    assert dense == pytest.approx(18.4e9, rel=0.01)


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert out.returncode == 2
    assert "one GPU" in out.stderr
    assert out.stdout.strip() == ""


def test_generation_counter_record_matches_generate_hip():
    rec = bench.counter_record("gen_1k", kind="generate")
    assert rec is not None, "profiles/generate_traffic_gen_1k.json was taken on another generate.hip"
    assert rec["traffic_bytes_per_launch"] > 0


@pytest.mark.parametrize("tag,workload,kernel", [("paper_hybrid1", "paper", "hybrid")])
def test_alternative_shape_records_describe_the_current_kernel(tag, workload, kernel):
    """Counter records of a workload in a shape other than its recorded one
    (profiles/render_traffic_<tag>.json, cited beside the bench line) are of
    the current render.hip too."""
    raw = json.load(open(os.path.join(ROOT, "profiles", f"render_traffic_{tag}.json")))
    src = open(os.path.join(ROOT, "paper_2204_02585_amd", "csrc", "render.hip"), "rb").read()
    assert raw["render_hip_sha256_16"] == hashlib.sha256(src).hexdigest()[:16]
    assert raw["workload"] == workload and kernel in raw["kernel"]
    assert raw["td_busy_cycles_per_launch"] <= 256 * 2.4e3 * raw["kernel_us_trace"]

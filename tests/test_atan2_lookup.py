"""Accuracy of the binary64 atan2 the render kernels use for the direction
lookup (csrc/atan2_lookup.h), built for the host with hipcc and compared with
numpy's arctan2.  The bilinear lookup of beta (Sec. 3.4) needs the angles to
about 1e-8; the function is specified to 2e-14."""
import os
import subprocess

import numpy as np
import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2204_02585_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

PROGRAM = r"""
#include <stdio.h>
#include "atan2_lookup.h"
int main(int argc, char** argv)
{
    FILE* in = fopen(argv[1], "rb");
    FILE* out = fopen(argv[2], "wb");
    double yx[2];
    while (fread(yx, sizeof(double), 2, in) == 2) {
        const double r = sqn::atan2_lookup(yx[0], yx[1]);
        fwrite(&r, sizeof(double), 1, out);
    }
    fclose(in);
    fclose(out);
    return 0;
}
"""


def _pairs():
    rng = np.random.Generator(np.random.PCG64(11))
    n = 200_000
    ang = rng.uniform(-np.pi, np.pi, n)
    mag = 10.0 ** rng.uniform(-30, 30, n)
    y, x = mag * np.sin(ang), mag * np.cos(ang)
    # near the octant and reduction boundaries: |y| ~ |x|, |y| ~ tan(pi/8)|x|
    t = np.tan(np.pi / 8)
    b = rng.uniform(-1e-9, 1e-9, 4000)
    extra = [(1.0 + b, np.ones_like(b)), (t * (1.0 + b), np.ones_like(b)),
             (np.ones_like(b), t * (1.0 + b)), (-(1.0 + b), np.ones_like(b))]
    ys = [y] + [e[0] for e in extra]
    xs = [x] + [e[1] for e in extra]
    special = np.array([(0.0, 1.0), (-0.0, 1.0), (0.0, -1.0), (-0.0, -1.0), (1.0, 0.0), (-1.0, 0.0),
                        (1.0, -0.0), (0.0, 0.0), (-0.0, 0.0), (0.0, -0.0), (-0.0, -0.0),
                        (1e-300, 1.0), (1.0, 1e-300), (-1.0, -1e300)])
    return np.concatenate([np.stack([np.concatenate(ys), np.concatenate(xs)], 1), special])


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc missing")
def test_atan2_lookup_accuracy(tmp_path):
    src = tmp_path / "atan2_check.hip"
    src.write_text(PROGRAM)
    exe = tmp_path / "atan2_check"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O2", "-ffp-contract=off", "-I", CSRC, "-o", str(exe),
                    str(src)], check=True, capture_output=True)
    yx = _pairs()
    (tmp_path / "in.bin").write_bytes(yx.astype(np.float64).tobytes())
    subprocess.run([str(exe), str(tmp_path / "in.bin"), str(tmp_path / "out.bin")], check=True)
    got = np.frombuffer((tmp_path / "out.bin").read_bytes(), dtype=np.float64)
    want = np.arctan2(yx[:, 0], yx[:, 1])
    assert got.shape == want.shape
    err = np.abs(got - want)
    assert float(err.max()) <= 2e-14, float(err.max())
    # signs and zeros as atan2: the signed zeros map to +-0 and +-pi
    assert np.array_equal(np.signbit(got), np.signbit(want))

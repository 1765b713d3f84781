"""The built render library's device code holds no packed binary32 VALU
forms (v_pk_add_f32, v_pk_mul_f32, v_pk_fma_f32): the build passes
-target-feature -packed-fp32-ops to the device compiler, and this test reads
the gfx950 code objects back out of libsqn.so and disassembles them."""
import os
import re
import struct
import subprocess

import pytest

from paper_2204_02585_amd import build

LLVM = "/opt/rocm/llvm/bin"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
PACKED_F32 = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")


def device_code_objects(lib_path, tmp):
    """The amdgcn entries of the clang offload bundles in the library's
    .hip_fatbin section (one bundle per source file)."""
    fatbin = os.path.join(tmp, "fatbin")
    subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fatbin}", lib_path,
                    os.path.join(tmp, "lib.stripped")], check=True)
    data = open(fatbin, "rb").read()
    objs, pos = [], 0
    while True:
        start = data.find(MAGIC, pos)
        if start < 0:
            return objs
        (n,) = struct.unpack_from("<Q", data, start + len(MAGIC))
        p = start + len(MAGIC) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", data, p)
            p += 24
            triple = data[p:p + tlen].decode()
            p += tlen
            if "amdgcn" in triple:
                objs.append((triple, data[start + off:start + off + size]))
        pos = start + len(MAGIC)


@pytest.mark.skipif(not os.path.exists(f"{LLVM}/llvm-objdump"), reason="ROCm llvm tools missing")
def test_no_packed_fp32_in_device_code(tmp_path):
    assert os.path.exists(build.LIB_PATH), "build the library first"
    objs = device_code_objects(build.LIB_PATH, str(tmp_path))
    assert len(objs) == len(build.SOURCES)
    kernels = 0
    for k, (triple, blob) in enumerate(objs):
        assert triple.endswith("gfx950")
        path = tmp_path / f"co{k}.o"
        path.write_bytes(blob)
        asm = subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", str(path)], check=True,
                             capture_output=True, text=True).stdout
        kernels += asm.count("s_endpgm")
        hits = PACKED_F32.findall(asm)
        assert not hits, f"{triple} object {k}: {len(hits)} packed binary32 instructions"
    # the disassembly did see the kernels
    assert kernels > 50

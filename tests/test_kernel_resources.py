"""No kernel in the built library spills registers to scratch memory.

The gfx950 code objects are read out of libnvfp4.so's offload bundles (the
library built here from this repository's sources) and each kernel's
metadata is checked: private segment size 0 and no VGPR spills.  (SGPR
spills, which the FP32-output GEMM variants have, go to lanes of a spare
VGPR when the private segment is empty: no memory traffic.)  A spilling
variant of the fused quantize + GEMM kernels once needed 208-220
bytes of scratch per lane; this test keeps every kernel off that path.
Needs no GPU."""

import os
import re
import shutil
import struct
import subprocess

import pytest

from paper_2609_04098_amd import nvfp4 as C

LLVM = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin")
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
DEVICE = "hipv4-amdgcn-amd-amdhsa--gfx950"
KEYS = ("private_segment_fixed_size", "vgpr_spill_count")


def device_objects(fat):
    """Yield the gfx950 code objects of each offload bundle in `fat`."""
    start = fat.find(MAGIC)
    while start >= 0:
        n = struct.unpack_from("<Q", fat, start + len(MAGIC))[0]
        q = start + len(MAGIC) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", fat, q)
            q += 24
            triple = fat[q:q + tlen].decode()
            q += tlen
            if triple == DEVICE and size:
                yield fat[start + off:start + off + size]
        start = fat.find(MAGIC, start + 1)


def kernel_metadata(readelf, path):
    """{kernel name: {key: int}} from the code object's metadata note."""
    text = subprocess.run([readelf, "--notes", path], check=True, capture_output=True, text=True).stdout
    out, cur = {}, None
    for line in text.splitlines():
        m = re.match(r"^    \.(\w+):\s+(\S+)", line)      # kernel-level keys (arguments are nested deeper)
        if not m:
            continue
        if m.group(1) == "name":
            cur = out.setdefault(m.group(2), {})
        elif cur is not None and m.group(1) in KEYS:
            cur[m.group(1)] = int(m.group(2))
    return out


def test_no_kernel_uses_scratch(tmp_path):
    objcopy, readelf = os.path.join(LLVM, "llvm-objcopy"), os.path.join(LLVM, "llvm-readelf")
    if not (os.path.exists(C.LIB_PATH) and shutil.which(objcopy) and shutil.which(readelf)):
        pytest.skip("library or LLVM tools not available")
    fat = tmp_path / "fat.bin"
    subprocess.run([objcopy, "--dump-section=.hip_fatbin=%s" % fat, C.LIB_PATH, str(tmp_path / "lib.so")],
                   check=True, capture_output=True)
    kernels = {}
    for i, co in enumerate(device_objects(fat.read_bytes())):
        p = tmp_path / ("dev%d.co" % i)
        p.write_bytes(co)
        kernels.update(kernel_metadata(readelf, str(p)))
    # every translation unit with kernels: quantizers, weight pack, GEMMs, fused paths
    assert len(kernels) >= 60, sorted(kernels)
    bad = {k: v for k, v in kernels.items() if set(v) != set(KEYS) or any(v.values())}
    assert not bad, bad

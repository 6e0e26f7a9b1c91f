"""No kernel in the built library spills registers to scratch memory.

The gfx950 code objects are read out of libnvfp4.so's offload bundles (the
library built here from this repository's sources), and each kernel's
entry in the AMDGPU metadata note (a MessagePack map) is checked: private
segment size 0 and no VGPR spills.  (SGPR spills, which the FP32-output GEMM
variants have, go to lanes of a spare VGPR when the private segment is
empty: no memory traffic.)  A spilling variant of the fused quantize + GEMM
kernels once needed 208-220 bytes of scratch per lane; this test keeps
every kernel off that path.  Plain ELF and bundle parsing, no tools and no
GPU."""

import os
import struct

import pytest

from paper_2609_04098_amd import nvfp4 as C

msgpack = pytest.importorskip("msgpack")

MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
DEVICE = "hipv4-amdgcn-amd-amdhsa--gfx950"
NT_AMDGPU_METADATA = 32


def elf_sections(b):
    """{name: bytes} of a little-endian ELF64 image."""
    assert b[:4] == b"\x7fELF" and b[4] == 2 and b[5] == 1, "not a little-endian ELF64 file"
    shoff = struct.unpack_from("<Q", b, 0x28)[0]
    shentsize, shnum, shstrndx = struct.unpack_from("<HHH", b, 0x3A)
    hdr = [struct.unpack_from("<IIQQQQIIQQ", b, shoff + i * shentsize) for i in range(shnum)]
    names = hdr[shstrndx][4]
    out = {}
    for h in hdr:
        name = b[names + h[0]: b.index(b"\0", names + h[0])].decode()
        out[name] = b[h[4]: h[4] + h[5]]
    return out


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


def kernel_metadata(code_object):
    """The `amdhsa.kernels` entries of a code object's metadata note."""
    note = elf_sections(code_object)[".note"]
    q, kernels = 0, []
    while q + 12 <= len(note):
        namesz, descsz, kind = struct.unpack_from("<III", note, q)
        q += 12 + ((namesz + 3) & ~3)
        desc = note[q:q + descsz]
        q += (descsz + 3) & ~3
        if kind == NT_AMDGPU_METADATA:
            kernels += msgpack.unpackb(desc, raw=False, strict_map_key=False)["amdhsa.kernels"]
    return kernels


def test_no_kernel_uses_scratch():
    if not os.path.exists(C.LIB_PATH):
        pytest.skip("library not built")
    fat = elf_sections(open(C.LIB_PATH, "rb").read())[".hip_fatbin"]
    kernels = [k for co in device_objects(fat) for k in kernel_metadata(co)]
    # every translation unit with kernels: quantizers, weight pack, GEMMs, fused paths
    assert len(kernels) >= 60, [k[".name"] for k in kernels]
    bad = {k[".name"]: (k[".private_segment_fixed_size"], k.get(".vgpr_spill_count"))
           for k in kernels if k[".private_segment_fixed_size"] != 0 or k.get(".vgpr_spill_count", 0) != 0}
    assert not bad, bad

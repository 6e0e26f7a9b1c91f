"""Build libnvfp4.so (the HIP kernels and the C ABI) in this directory for
gfx950 with hipcc.  Run as ``python -m paper_2609_04098_amd.build_lib``
(``--incremental`` reuses the objects of unchanged sources from
``_build/``, keyed by a hash of the source, every header and the flags)."""

import glob
import hashlib
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnvfp4.so")
OBJ_CACHE = os.path.join(HERE, "_build")

SOURCES = ["api.cpp", "act_quant.hip", "norm_quant.hip", "weight_pack.hip", "gemm.hip", "gemm_lds_square.hip",
           "gemm_lds_super.hip", "gemm_lds_super_f32.hip", "gemm_lds_tall.hip", "gemm_splitk.hip", "gemm_reg.hip",
           "quant_gemm.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # Quantization decisions rely on single roundings where written; no
    # implicit contraction of a * b + c.
    "-ffp-contract=off",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    # Packed FP32 instructions are not generated.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _key(src):
    """Hash of one source, every header it may include, and the flags."""
    h = hashlib.sha256(" ".join(HIPCC_FLAGS).encode())
    for p in [os.path.join(CSRC, src)] + sorted(glob.glob(os.path.join(CSRC, "*.h"))) + \
            sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        with open(p, "rb") as f:
            h.update(p.encode() + f.read())
    return h.hexdigest()[:20]


def build(verbose=False, incremental=False):
    """Compile every source to an object (in parallel), then link the shared
    library atomically (write to a temporary file, then rename)."""
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    tmpdir = tempfile.mkdtemp(prefix="nvfp4_build_")
    if incremental:
        os.makedirs(OBJ_CACHE, exist_ok=True)
    procs, objs, cached = [], [], []
    for src in SOURCES:
        obj = os.path.join(tmpdir, src.replace(".", "_") + ".o")
        if incremental:
            keep = os.path.join(OBJ_CACHE, "%s.%s.o" % (src.replace(".", "_"), _key(src)))
            if os.path.exists(keep):
                objs.append(keep)
                continue
            cached.append((obj, keep))
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [hipcc()] + HIPCC_FLAGS + inc + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = False
    for cmd, p in procs:
        out, _ = p.communicate()
        text = "\n".join(l for l in out.decode(errors="replace").splitlines()
                         if "packed-fp32-ops' is not a recognized feature" not in l)
        if p.returncode != 0:
            failed = True
            sys.stderr.write(" ".join(cmd) + "\n" + text + "\n")
        elif verbose and text.strip():
            sys.stderr.write(text + "\n")
    if failed:
        raise RuntimeError("hipcc failed building libnvfp4.so")
    tmp_lib = LIB + ".tmp%d" % os.getpid()
    link = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp_lib] + objs
    r = subprocess.run(link, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        sys.stderr.write(r.stdout.decode(errors="replace"))
        raise RuntimeError("hipcc link of libnvfp4.so failed")
    os.replace(tmp_lib, LIB)
    for obj, keep in cached:
        stem = os.path.basename(keep).split(".")[0]
        for old in glob.glob(os.path.join(OBJ_CACHE, stem + ".*.o")):
            os.remove(old)
        os.replace(obj, keep)
    for o in os.listdir(tmpdir):
        os.remove(os.path.join(tmpdir, o))
    os.rmdir(tmpdir)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True, incremental="--incremental" in sys.argv[1:]))

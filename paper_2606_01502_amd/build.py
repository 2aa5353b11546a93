"""Build libmla_sparse.so (HIP, gfx950) in-tree with hipcc.

Each csrc/*.hip file is compiled separately (in parallel) and linked into
paper_2606_01502_amd/libmla_sparse.so.  Packed-FP32 instructions are
disabled for every device compile.  The device assembly of every source is
generated beside the objects and checked for matrix-core wait-state hazards
around the inline-asm products (hazards.py); a hazard fails the build.
"""
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmla_sparse.so")
BUILD_DIR = os.path.join(ROOT, "_build")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _compile(src, extra=()):
    os.makedirs(BUILD_DIR, exist_ok=True)
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{p.stderr}")
    return obj


def _device_asm(src, extra=()):
    os.makedirs(BUILD_DIR, exist_ok=True)
    out = os.path.join(BUILD_DIR, os.path.basename(src) + ".s")
    cmd = [HIPCC, *FLAGS, *extra, "--cuda-device-only", "-S", src, "-o", out]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{p.stderr}")
    return out


def check_hazards(asm_files):
    """Raise if the device assembly has a wait-state hazard (see hazards.py)."""
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    from paper_2606_01502_amd import hazards
    bad = []
    for f in asm_files:
        with open(f) as fh:
            bad += [f"{os.path.basename(f)}: {v}" for v in hazards.check(fh.read())]
    if bad:
        raise RuntimeError("matrix-core wait-state hazards in the device code:\n" +
                           "\n".join(bad[:20]))


def build(extra=(), out=LIB):
    """Compile every csrc/*.hip for gfx950, check the device assembly for
    wait-state hazards and link the shared library."""
    srcs = sources()
    with ThreadPoolExecutor(max_workers=min(8, 2 * len(srcs))) as ex:
        obj_jobs = [ex.submit(_compile, s, extra) for s in srcs]
        asm_jobs = [ex.submit(_device_asm, s, extra) for s in srcs]
        objs = [j.result() for j in obj_jobs]
        asms = [j.result() for j in asm_jobs]
    check_hazards(asms)
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"link failed:\n{p.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(sys.argv[1:]))

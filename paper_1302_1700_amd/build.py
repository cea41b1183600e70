"""Build libfragscan.so and libfragscan_debug.so (HIP, gfx950) in-tree.

    python -m paper_1302_1700_amd.build        # or: python paper_1302_1700_amd/build.py

Each .hip source is compiled to an object under _build/ (in parallel), then
linked into paper_1302_1700_amd/libfragscan.so; the same sources compiled
with -DFRAGSCAN_DEBUG (objects under _build/debug/) make
libfragscan_debug.so, whose kernels check every fragment access against the
true fragment sizes and whose scans return FS_ERR_BOUNDS when a check fails.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libfragscan.so")
LIB_DEBUG = os.path.join(HERE, "libfragscan_debug.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result", "-I", os.path.join(ROOT, "include")]
# accumulate matrix-core products in ordinary VGPRs (no AGPR copies); the
# *_wide.hip register tiles need the accumulation registers and go without
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src, quiet, debug=False):
    obj = os.path.join(BUILD, "debug" if debug else "", os.path.basename(src)[:-4] + ".o")
    form = [] if src.endswith("_wide.hip") else VGPR_FORM
    cmd = [HIPCC] + FLAGS + form + (["-DFRAGSCAN_DEBUG"] if debug else []) + ["-c", src, "-o", obj]
    if not quiet:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s\n%s" % (src, r.stdout, r.stderr))
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    if msgs and not quiet:
        print(msgs, flush=True)
    return obj


def _link(objs, lib, quiet):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if not quiet:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, lib)


def build(quiet=False, jobs=None, debug=True):
    """Both libraries (debug=False: the release one only)."""
    os.makedirs(os.path.join(BUILD, "debug"), exist_ok=True)
    srcs = sources()
    units = [(s, False) for s in srcs] + ([(s, True) for s in srcs] if debug else [])
    jobs = jobs or min(len(units), max(1, min(os.cpu_count() or 1, 16)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda u: _compile(u[0], quiet, u[1]), units))
    _link(objs[:len(srcs)], LIB, quiet)
    if debug:
        _link(objs[len(srcs):], LIB_DEBUG, quiet)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)

"""The library's host planner and the C oracle under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

The planner: every HIP source compiled with the sanitizers on the host code only
(the device code is built as usual and never run), linked with
tests/sanitize/planner_main.cpp,
which drives the planning-only paths of the C-ABI on the workload nets and
300 seeded random stacks.  The oracle: patch_oracle.c with gcc and the same
sanitizers, driven by tests/sanitize/oracle_main.c on small nets.  Any
sanitizer report fails the run (halt_on_error)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = {"ASAN_OPTIONS": "halt_on_error=1:detect_leaks=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-3000:], r.stderr[-3000:])
    return r


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_planner_under_sanitizers(tmp_path):
    import concurrent.futures as cf
    csrc = os.path.join(ROOT, "paper_1302_1700_amd", "csrc")
    srcs = sorted(os.path.join(csrc, f) for f in os.listdir(csrc) if f.endswith(".hip"))
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all"]
    # device code unoptimised: it is never run here, and builds twice as fast
    flags = ["--offload-arch=gfx950", "-O1", "-Xarch_device", "-O0", "-g", "-std=c++17", "-fno-omit-frame-pointer",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include")] + san

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC] + flags + ["-c", src, "-o", obj])
        return obj

    with cf.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, srcs + [os.path.join(ROOT, "tests", "sanitize", "planner_main.cpp")]))
    exe = str(tmp_path / "planner_san")
    _run([HIPCC, "--offload-arch=gfx950", "-o", exe] + objs + san)
    env = dict(os.environ, **SAN_ENV)
    r = _run([exe], env=env, timeout=600)
    assert "0 failures" in r.stdout, r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-O1", "-g", "-std=c99", "-fopenmp", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-fno-omit-frame-pointer", "-o", exe, os.path.join(ROOT, "oracle", "patch_oracle.c"),
          os.path.join(ROOT, "tests", "sanitize", "oracle_main.c"), "-lm"])
    env = dict(os.environ, OMP_NUM_THREADS="2", **SAN_ENV)
    r = _run([exe], env=env, timeout=600)
    assert "oracle sanitizer run ok" in r.stdout, r.stdout

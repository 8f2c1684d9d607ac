"""The host side of the C ABI (wm_api.cpp, wm_profile.cpp) built with
AddressSanitizer + UndefinedBehaviorSanitizer, and with ThreadSanitizer, and
driven on the CPU by tests/sanitize/abi_driver.cpp: argument validation of
every entry point, the size queries (including sizes that would overflow),
the no-op paths, the profile registry, and per-thread error strings from
eight threads at once.  No call reaches the GPU.

The sanitizers instrument host code only: each -fsanitize= on a hipcc line
follows -Xarch_host, so no device code is built with them; the link line is
the host compiler's.  The kernel objects come from the library build."""

import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2205_01435_amd")
BUILD = os.path.join(PKG, "_build")
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"
HOST_SOURCES = [os.path.join(PKG, "csrc", "wm_api.cpp"), os.path.join(PKG, "csrc", "wm_profile.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp")]

pytestmark = pytest.mark.skipif(
    not (os.path.exists(HIPCC) and os.path.exists(CLANG) and glob.glob(os.path.join(BUILD, "wm_kernels.o"))),
    reason="needs hipcc and the library's object files (run __graft_entry__.build())")


def _build(tmp_path, sanitizers):
    flags = ["-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
             "-Xarch_host", "-fno-omit-frame-pointer"]
    for s in sanitizers:
        flags += ["-Xarch_host", f"-fsanitize={s}"]
    objs = []
    for src in HOST_SOURCES:
        o = str(tmp_path / (os.path.splitext(os.path.basename(src))[0] + ".o"))
        subprocess.run([HIPCC, *flags, "-c", src, "-o", o], check=True, capture_output=True, text=True)
        objs.append(o)
    kernels = [o for o in sorted(glob.glob(os.path.join(BUILD, "*.o")))
               if os.path.basename(o) not in ("wm_api.o", "wm_profile.o")]
    exe = str(tmp_path / "driver")
    subprocess.run([CLANG, "-fsanitize=" + ",".join(sanitizers), *objs, *kernels, "-L/opt/rocm/lib",
                    "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe], check=True, capture_output=True,
                   text=True)
    return exe


def _run(exe, *args, env_extra):
    env = dict(os.environ, HIP_VISIBLE_DEVICES="", **env_extra)
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    for marker in ("ERROR: AddressSanitizer", "runtime error:", "WARNING: ThreadSanitizer"):
        assert marker not in out, out[-4000:]
    assert "0 failures" in r.stdout


def test_abi_under_address_and_undefined_sanitizers(tmp_path):
    exe = _build(tmp_path, ["address", "undefined"])
    # leaks of the HIP runtime's own one-time allocations are not this code's
    _run(exe, env_extra={"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0",
                         "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})


def test_abi_under_thread_sanitizer(tmp_path):
    exe = _build(tmp_path, ["thread"])
    _run(exe, "threads", env_extra={"TSAN_OPTIONS": "halt_on_error=1"})

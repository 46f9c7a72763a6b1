"""The C ABI's host side under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Every library source is compiled with the sanitizers on its host side only (the GPU
code is unchanged), linked with the driver tests/abi_validate.cpp, and run: the
host-only entry points on valid and invalid input, every device entry point's
argument validation, extreme sizes, and valid calls up to the device check.  Any
sanitizer report aborts the driver.  The instrumented build is kept under
_build/sanitize/ and redone when a source changes.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2405_19509_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(ROOT, "_build", "sanitize")
DRIVER = os.path.join(ROOT, "tests", "abi_validate.cpp")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = ["address", "undefined"]
HOST_SAN = [f for s in SAN for f in ("-Xarch_host", f"-fsanitize={s}")] + \
    ["-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def _stamp():
    h = hashlib.sha256()
    for f in _sources() + sorted(glob.glob(os.path.join(CSRC, "*.h"))) + [os.path.join(INCLUDE, "gcx.h"), DRIVER,
                                                                          os.path.abspath(__file__)]:
        h.update(f.encode())
        h.update(open(f, "rb").read())
    return h.hexdigest()


def _compile(src):
    obj = os.path.join(OUT, os.path.basename(src) + ".o")
    cmd = [HIPCC, "-x", "hip", "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-I", INCLUDE,
           "-I", CSRC, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wno-unused-command-line-argument", *HOST_SAN, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed for {src}:\n{r.stderr[-3000:]}")
    return obj


def _build():
    exe = os.path.join(OUT, "abi_validate")
    stamp = os.path.join(OUT, "stamp")
    want = _stamp()
    if os.path.exists(exe) and os.path.exists(stamp) and open(stamp).read() == want:
        return exe
    shutil.rmtree(OUT, ignore_errors=True)
    os.makedirs(OUT)
    srcs = _sources()
    with cf.ThreadPoolExecutor(max(1, min(8, len(srcs)))) as ex:
        objs = list(ex.map(_compile, srcs))
    drv = os.path.join(OUT, "abi_validate.o")
    hip_inc = ["-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include"]
    san = "-fsanitize=" + ",".join(SAN)
    r = subprocess.run([CLANG, "-O1", "-g", "-std=c++17", "-I", INCLUDE, *hip_inc, san, "-c", DRIVER, "-o", drv],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([CLANG, san, drv, *objs, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
                        "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    open(stamp, "w").write(want)
    return exe


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not found")
def test_abi_host_side_under_sanitizers():
    exe = _build()
    env = dict(os.environ)
    # the HIP runtime keeps allocations for the process lifetime: leaks are not this test's subject
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["HIP_VISIBLE_DEVICES"] = ""  # no device: valid device calls stop at the device check
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-2000:] + r.stderr[-4000:]

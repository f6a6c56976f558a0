"""The host runtime of the C ABI under AddressSanitizer, LeakSanitizer and
UBSan, on the CPU: the library's sources are rebuilt with the sanitizers on
the host code only (device code is compiled as usual), linked into a small
driver (tests/host/abi_checks.cpp) that exercises configuration checks,
layouts, workspace plans, the argument checks of every entry point and the
error paths that reach the HIP runtime without a device. Any memory error,
leak or undefined behaviour aborts the driver."""
import hashlib
import os
import shutil
import subprocess
import concurrent.futures as cf

import pytest

from paper_2609_37029_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST = os.path.join(ROOT, "tests", "host")
OUT = os.path.join(HOST, "_build")
CLANG = "/opt/rocm/llvm/bin/clang++"
ROCM_LIB = "/opt/rocm/lib"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def _digest():
    h = hashlib.sha256()
    for f in sorted(B.SOURCES) + ["ldr_internal.h", "noise.h"]:
        h.update(open(os.path.join(B.CSRC, f), "rb").read())
    for f in (os.path.join(ROOT, "include", "ldr.h"), os.path.join(HOST, "abi_checks.cpp")):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def _build():
    exe = os.path.join(OUT, "abi_checks")
    stamp = os.path.join(OUT, "stamp")
    dig = _digest()
    if os.path.exists(exe) and os.path.exists(stamp) and open(stamp).read() == dig:
        return exe
    os.makedirs(OUT, exist_ok=True)
    hipcc = B.hipcc()

    def obj(src):
        o = os.path.join(OUT, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc] + B.flags() + SAN + ["-x", "hip", "-c", os.path.join(B.CSRC, src), "-o", o]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        return o
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(obj, B.SOURCES))
    # the driver is host code only: plain clang++, linked against the HIP runtime
    drv = os.path.join(OUT, "abi_checks.o")
    host_san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                "-fno-omit-frame-pointer", "-g"]
    r = subprocess.run([CLANG, "-O1", "-std=c++17"] + host_san +
                       ["-I", os.path.join(ROOT, "include"), "-c",
                        os.path.join(HOST, "abi_checks.cpp"), "-o", drv],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([CLANG] + host_san + ["-o", exe, drv] + objs +
                       ["-L", ROCM_LIB, "-lamdhip64", "-Wl,-rpath," + ROCM_LIB],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    open(stamp, "w").write(dig)
    return exe


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc is required to build the sanitized library")
def test_host_runtime_under_asan_and_ubsan():
    exe = _build()
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:verify_asan_link_order=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["HIP_VISIBLE_DEVICES"] = ""       # host paths only, also on a machine with a GPU
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "abi checks ok" in r.stdout

"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU).

The library sources are compiled as usual for gfx950 but with the
sanitizers on the host side only (each flag behind -Xarch_host), linked with
tests/abi_host_driver.cpp, and run: argument and shape errors of every entry
point, workspace-size queries over extreme sizes (up to INT32_MAX tokens),
the streamed layer's ring schedule on 512 configurations, the status
strings.  The run must end with every call returning its expected status
and without a sanitizer report (heap or stack overflow, leak, signed
overflow, null or misaligned access).  The `enum` check is off: the ABI is C,
where an enum parameter may carry any int, and the library range-checks it.
About 15 s of compile time on 8 cores.
"""
import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_10493_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize=enum", "-Xarch_host", "-fno-sanitize-recover=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr}"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_host_abi_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", *SAN,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-fhip-fp32-correctly-rounded-divide-sqrt", "-I", INCLUDE, "-I", CSRC]
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    objs = [str(tmp_path / (os.path.basename(s) + ".o")) for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        list(ex.map(_run, [[HIPCC, *flags, "-c", s, "-o", o] for s, o in zip(srcs, objs)]))
    drv = str(tmp_path / "driver.o")
    _run([HIPCC, "-x", "c++", "-O1", "-g", "-std=c++17", *SAN, "-I", INCLUDE, "-I", "/opt/rocm/include",
          "-D__HIP_PLATFORM_AMD__", "-c", os.path.join(ROOT, "tests", "abi_host_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_host_driver")
    _run([HIPCC, "--offload-arch=gfx950", *SAN, *objs, drv, "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "ERROR: AddressSanitizer" not in out and "LeakSanitizer" not in out
    assert " 0 failures" in out

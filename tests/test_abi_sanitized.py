"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Every source file is compiled again with the sanitizers on its host code
only (the device code is built as usual, never run), linked with the check
program ``abi_host_check.cpp``, which calls every entry point with
arguments that fail validation and every workspace query across extreme
sizes, and run on the CPU: a sanitizer report aborts it.  No GPU is used.
"""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1912_06680_amd", "csrc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-w",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return None


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(" ".join(cmd) + "\n" + res.stdout[-4000:] + res.stderr[-4000:])


@pytest.mark.slow
def test_abi_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not found")
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    objs = [str(tmp_path / (s[:-4] + ".o")) for s in srcs]
    with cf.ThreadPoolExecutor(min(8, len(srcs))) as ex:
        futs = [ex.submit(_run, [hipcc, *FLAGS, *SAN, "-c", os.path.join(CSRC, s), "-o", o])
                for s, o in zip(srcs, objs)]
        for f in futs:
            f.result()
    drv = str(tmp_path / "abi_host_check.o")
    _run([hipcc, "-O1", "-g", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"),
          "-c", os.path.join(ROOT, "tests", "abi_host_check.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_host_check")
    _run([hipcc, "--offload-arch=gfx950", *SAN, *objs, drv, "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-6000:]
    assert "all" in res.stdout and "checks passed" in res.stdout, out[-2000:]

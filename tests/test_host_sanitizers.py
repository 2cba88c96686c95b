"""The library's host API sources built with AddressSanitizer and UBSan and
driven on the CPU.

`tests/sanitize/hip_stub.cpp` stands in for the HIP runtime (host memory,
memcpy, no-op events and streams) and for the kernel launchers (they check the
parameters the host side hands a kernel, and count the launch);
`tests/sanitize/driver.cpp` calls every entry point of the attention, fusion
and projected-KV handles with valid and invalid arguments, plans, forced
paths and split counts, the no-allocation call, validation, and more calls
than the profiling rings hold.  The three host sources are compiled for the
host only (no device code), with each -fsanitize= flag placed after
-Xarch_host, so nothing GPU-side is instrumented.

Command (what `build_and_run` does), from the repository root:
  hipcc -x hip --cuda-host-only -O1 -g -std=c++17 -fno-omit-frame-pointer -I include -I paper_2604_26412_amd/csrc
        -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -c <each of api.cpp fusion_api.cpp
        kvproj_api.cpp tests/sanitize/hip_stub.cpp>
  clang++ -fsanitize=address,undefined -c tests/sanitize/driver.cpp; clang++ -fsanitize=address,undefined *.o
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_26412_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


def build_and_run(out_dir):
    flags = ["-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
             "-Wno-unused-command-line-argument"]
    san_host = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=undefined"]
    objs = []
    sources = [os.path.join(CSRC, f) for f in ("api.cpp", "fusion_api.cpp", "kvproj_api.cpp")]
    sources.append(os.path.join(SAN, "hip_stub.cpp"))
    for src in sources:
        obj = os.path.join(out_dir, os.path.basename(src) + ".o")
        _run([HIPCC, "-x", "hip", "--cuda-host-only", *flags, *san_host, "-c", src, "-o", obj])
        objs.append(obj)
    obj = os.path.join(out_dir, "driver.o")
    _run([CLANG, *flags, "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-c",
          os.path.join(SAN, "driver.cpp"), "-o", obj])
    objs.append(obj)
    # a host-only object that holds __device__ variables still names its (absent) device image
    names = set()
    for o in objs:
        for line in _run(["nm", "-u", o]).stdout.splitlines():
            m = re.search(r"\b(__hip_fatbin_[0-9a-f]+)\b", line)
            if m:
                names.add(m.group(1))
    stub = os.path.join(out_dir, "fatbin_names.c")
    with open(stub, "w") as f:
        for n in sorted(names):
            f.write(f"const char {n}[16] = {{0}};\n")
    obj = os.path.join(out_dir, "fatbin_names.o")
    _run([CLANG, "-x", "c", "-c", stub, "-o", obj])
    objs.append(obj)
    exe = os.path.join(out_dir, "host_api_driver")
    _run([CLANG, "-fsanitize=address,undefined", *objs, "-o", exe, "-lpthread", "-lm"])
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    return subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG) and shutil.which("nm")),
                    reason="ROCm compilers not installed")
def test_host_api_is_clean_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    r = build_and_run(str(tmp_path))
    report = r.stdout + r.stderr
    assert "AddressSanitizer" not in report and "LeakSanitizer" not in report, report[-6000:]
    assert "runtime error" not in report, report[-6000:]
    assert r.returncode == 0, report[-6000:]
    m = re.search(r"launches (\d+), bad launch parameters (\d+), failed expectations (\d+)", r.stdout)
    assert m and int(m.group(1)) > 1000 and m.group(2) == "0" and m.group(3) == "0", r.stdout

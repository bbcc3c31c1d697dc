"""The library's host code (planner, page allocator, runtime argument checks) under
AddressSanitizer and UndefinedBehaviorSanitizer: tests/host/sanitize_driver.cpp drives the
C ABI with thousands of random plans, placements, maps, page reservations and context
descriptors, every runtime call being one that must be rejected before any device work.
The host sources are compiled here with the sanitizers (runtime.cpp through hipcc, host
side only) and linked with the library's device-kernel objects; CPU only."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_15943_amd", "csrc")
INC = os.path.join(ROOT, "include")
OUT = os.path.join(ROOT, "_build", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang++"
HIPCC = "/opt/rocm/bin/hipcc"
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


def test_host_code_under_address_and_ub_sanitizers():
    if not (os.path.exists(CLANG) and os.path.exists(HIPCC)):
        pytest.skip("ROCm clang / hipcc not installed")
    from paper_2608_15943_amd import build as b
    hip_objs = [os.path.join(b.BUILD, s + ".o") for s in b.HIP_SOURCES]
    if not all(os.path.exists(o) for o in hip_objs):
        b.build()
    os.makedirs(OUT, exist_ok=True)
    objs = []
    for src, extra in (("planner.cpp", ["-ffp-contract=off"]), ("pager.cpp", [])):
        o = os.path.join(OUT, src + ".o")
        _run([CLANG, "-O1", "-g", "-std=c++17", *SAN, *extra, "-I", INC, "-I", CSRC, "-c",
              os.path.join(CSRC, src), "-o", o])
        objs.append(o)
    o = os.path.join(OUT, "runtime.cpp.o")
    _run([HIPCC, "-O1", "-g", "-std=c++17", "--cuda-host-only", "-fno-omit-frame-pointer",
          "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-Xarch_host", "-fno-sanitize-recover=undefined", "-I", INC, "-I", CSRC, "-c",
          os.path.join(CSRC, "runtime.cpp"), "-o", o])
    objs.append(o)
    d = os.path.join(OUT, "driver.o")
    _run([CLANG, "-O1", "-g", "-std=c++17", *SAN, "-I", INC, "-c",
          os.path.join(ROOT, "tests", "host", "sanitize_driver.cpp"), "-o", d])
    exe = os.path.join(OUT, "sanitize_driver")
    _run([CLANG, *SAN, "-o", exe, d, *objs, *hip_objs, "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,/opt/rocm/lib"])
    env = dict(os.environ, ASAN_OPTIONS="halt_on_error=1:detect_leaks=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stderr
    assert "host checks passed" in r.stdout
    for bad in ("AddressSanitizer", "runtime error", "LeakSanitizer"):
        assert bad not in r.stderr, r.stderr

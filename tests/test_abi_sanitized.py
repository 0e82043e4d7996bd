"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer, on
the CPU.  The library's sources are compiled host-only with both sanitizers and
linked against a stand-in HIP runtime (tests/asan/hip_stub.cpp: one gfx950
device, host-malloc'd device memory, launches that only check their shape); a
driver (tests/asan/abi_driver.cpp) exercises every entry point's error paths and
valid calls.  Any memory error, leak or undefined behaviour in the host code, a
wrong status, an empty message, a launch shape outside the device's limits, a
HIP event or workspace not released fails the test."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_00051_amd", "csrc")
ASAN = os.path.join(ROOT, "tests", "asan")
SOURCES = ["api", "sampler", "disc_f32", "disc_bf16", "generator", "optim"]
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    if r.returncode != 0:
        raise AssertionError(f"{' '.join(cmd[:3])} ... failed:\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}")
    return r


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="hipcc / clang++ unavailable")
def test_abi_host_code_under_sanitizers(tmp_path):
    objs = []
    for s in SOURCES:
        o = str(tmp_path / f"{s}.o")
        _run([HIPCC, "--cuda-host-only", "-x", "hip", "-std=c++17", "-O1", "-g", "-fPIC", *SAN,
              "-c", os.path.join(CSRC, f"{s}.hip"), "-o", o])
        objs.append(o)
    # the fat-binary symbols the host-only objects refer to: empty stand-ins
    undef = _run(["nm", "-u", *objs]).stdout
    fat = sorted(set(re.findall(r"\b(__hip_fatbin_[0-9a-f]+)\b", undef)))
    fat_src = tmp_path / "fatbins.cpp"
    fat_src.write_text("".join(f'extern "C" const unsigned char {n}[16] = {{0}};\n' for n in fat))
    flags = ["-std=c++17", "-O1", "-g", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
             "-I" + os.path.join(ROOT, "include"), "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-fno-omit-frame-pointer"]
    extra = []
    for src in (os.path.join(ASAN, "hip_stub.cpp"), os.path.join(ASAN, "abi_driver.cpp"), str(fat_src)):
        o = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([CLANG, *flags, "-c", src, "-o", o])
        extra.append(o)
    exe = str(tmp_path / "abi_driver")
    _run([CLANG, "-fsanitize=address,undefined", *objs, *extra, "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:allocator_may_return_null=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout[-3000:])
    assert r.returncode == 0, f"driver failed ({r.returncode}):\n{r.stdout[-3000:]}\n{r.stderr[-6000:]}"
    assert "ALL OK" in r.stdout

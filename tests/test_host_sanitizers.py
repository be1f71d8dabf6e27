"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds the C ABI library's sources with the sanitizers on the host side
(`-Xarch_host -fsanitize=...`: the device code is compiled as usual and never
runs here), links them with the driver tests/host_sanitize/abi_checks.cpp,
and runs the segment validator (hand cases and 20000 random arrays) and the
argument checks of every entry point. No kernel is launched: every call the
driver makes fails a host check before the library touches a device.
"""

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2408_00539_amd", "csrc")
DRIVER = os.path.join(ROOT, "tests", "host_sanitize", "abi_checks.cpp")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
       "-fno-omit-frame-pointer"]


def _tools():
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    clangxx = "/opt/rocm/llvm/bin/clang++"
    if not (os.path.exists(hipcc) and os.path.exists(clangxx)):
        pytest.skip("ROCm toolchain not found")
    return hipcc, clangxx


def _host_san(flags):
    out = []
    for f in flags:
        out += ["-Xarch_host", f]
    return out


@pytest.mark.timeout(900)
def test_host_code_under_asan_and_ubsan(tmp_path):
    hipcc, clangxx = _tools()
    inc = ["-I" + os.path.join(ROOT, "include")]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        if src.endswith(".hip"):
            cmd = [hipcc, "--offload-arch=gfx950", "-std=c++17", "-O1", "-g", "-fPIC",
                   "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                   *_host_san(SAN), *inc, "-c", src, "-o", obj]
        else:
            cmd = [clangxx, "-std=c++17", "-O1", "-g", "-fPIC", *SAN, *inc, "-c", src,
                   "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj

    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) +
                  glob.glob(os.path.join(CSRC, "*.cpp"))) + [DRIVER]
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, srcs))
    exe = str(tmp_path / "abi_checks")
    r = subprocess.run([clangxx, *SAN, "-o", exe, *objs, "-L/opt/rocm/lib", "-lamdhip64",
                        "-Wl,-rpath,/opt/rocm/lib"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=23",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout[-2000:], r.stderr[-4000:])
    assert r.returncode == 0, r.stderr[-4000:]
    assert "host ABI checks passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr

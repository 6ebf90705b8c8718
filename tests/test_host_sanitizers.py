"""The library's host code (argument checks, plans, workspace sizing) built
with AddressSanitizer and UndefinedBehaviorSanitizer, driven through the C ABI
by tests/abi_host_check.c on the CPU. Only the host side of each source is
instrumented (device code is built as usual); every call in the driver
returns before anything is launched, so no GPU is needed."""

import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# the host compiler of that toolchain (one sanitizer runtime for every object)
CLANG = "/opt/rocm/llvm/bin/clang"
# host-only sanitizer flags: -Xarch_host right before each -fsanitize=
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


@pytest.mark.skipif(shutil.which(HIPCC) is None and not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_host_paths_under_asan_and_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2607_29591_amd", "csrc")
    inc = os.path.join(ROOT, "include")
    objs, procs = [], []
    for src in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.cpp"))):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        cmd = [HIPCC, "-O1", "-g", "-fPIC", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", *HOST_SAN, "-I", inc, "-c", src, "-o", obj]
        if src.endswith(".cpp"):
            cmd = [HIPCC, "-O1", "-g", "-fPIC", "-std=c++17", "--offload-arch=gfx950", *HOST_SAN, "-I", inc, "-x", "hip",
                   "-c", src, "-o", obj]
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
        objs.append(obj)
    for p in procs:
        out, _ = p.communicate(timeout=600)
        assert p.returncode == 0, out
    drv = str(tmp_path / "abi_host_check.o")
    subprocess.run([CLANG, "-O1", "-g", "-fPIC", "-fsanitize=address,undefined", "-I", inc, "-c",
                    os.path.join(ROOT, "tests", "abi_host_check.c"), "-o", drv], check=True)
    exe = str(tmp_path / "abi_host_check")
    link = subprocess.run([CLANG + "++", "-fsanitize=address,undefined", drv, *objs, "-L/opt/rocm/lib", "-lamdhip64",
                           "-Wl,-rpath,/opt/rocm/lib", "-o", exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                          text=True)
    assert link.returncode == 0, link.stdout
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout
    assert "abi host check: ok" in run.stdout
    assert "runtime error" not in run.stdout and "AddressSanitizer" not in run.stdout

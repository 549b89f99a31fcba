"""The C ABI's host-side paths under AddressSanitizer and UndefinedBehaviorSanitizer.

The runtime (every ABI entry point, configuration and argument checks, workspace carving,
size and FLOP queries) is compiled with both sanitizers on its host code and linked with
the kernels' objects of the regular build into `host_sanitizer_driver.cpp`, which
exercises every check that ends on the host.  Any memory error or undefined behaviour
aborts the driver."""

import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2408_07802_amd", "csrc")
BUILD = os.path.join(ROOT, "paper_2408_07802_amd", "_build")
HIPCC = "/opt/rocm/bin/hipcc"
CXX = "/opt/rocm/llvm/bin/clang++"
KERNEL_OBJECTS = ["norm", "gemm", "attention", "decode"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.skipif(not all(os.path.exists(os.path.join(BUILD, f + ".o")) for f in KERNEL_OBJECTS),
                    reason="the library is not built (run __graft_entry__.build())")
def test_host_paths_under_asan_and_ubsan(tmp_path):
    runtime = tmp_path / "runtime.o"
    # the sanitizers go on the host compilation only (-Xarch_host before each)
    comp = subprocess.run(
        [HIPCC, "-std=c++17", "-O1", "-g", "-fPIC", "--offload-arch=gfx950",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
         "-I" + os.path.join(ROOT, "include"), "-c", os.path.join(CSRC, "runtime.hip"),
         "-o", str(runtime)], capture_output=True, text=True)
    assert comp.returncode == 0, comp.stdout[-3000:] + comp.stderr[-3000:]
    # the driver is plain C++ (host compiler, sanitizers on), linked with the HIP runtime
    exe = tmp_path / "driver"
    link = subprocess.run(
        [CXX, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         "-I" + os.path.join(ROOT, "include"),
         os.path.join(ROOT, "tests", "host_sanitizer_driver.cpp")] +
        [str(runtime)] + [os.path.join(BUILD, f + ".o") for f in KERNEL_OBJECTS] +
        ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)],
        capture_output=True, text=True)
    assert link.returncode == 0, link.stdout[-3000:] + link.stderr[-3000:]
    env = dict(os.environ)
    # the HIP runtime's own allocations at exit are not this library's to report
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    run = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout[-3000:] + run.stderr[-5000:]
    assert "host paths clean" in run.stdout

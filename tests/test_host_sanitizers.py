"""The library's host code (validation, grouping, planner, scheduler) and the oracle
built with AddressSanitizer and UndefinedBehaviorSanitizer, exercised on
random batches by tests/sanitize/host_check.cpp.  CPU only: nothing is
launched on a GPU (the device code is compiled as usual and never run)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2401_11240_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang"
CLANGXX = "/opt/rocm/llvm/bin/clang++"
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not all(os.path.exists(c) for c in (HIPCC, CLANG, CLANGXX)), reason="ROCm compilers missing")
def test_planner_and_oracle_under_asan_ubsan(tmp_path):
    from paper_2401_11240_amd import build as B
    objs = []
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
    # the oracle: plain C, no OpenMP here (its pragmas are then ignored)
    objs.append(str(tmp_path / "oracle.o"))
    subprocess.run([CLANG, "-c", "-O1", "-g", "-std=c11", "-ffp-contract=off"] + san +
                   [os.path.join(ROOT, "oracle", "lora_oracle.c"), "-o", objs[-1]], check=True)
    # the library's host code and the driver (HIP sources: sanitizers on the
    # host side only; the driver stands in for the launch functions)
    host_san = []
    for f in san:
        host_san += ["-Xarch_host", f]
    for src in (os.path.join(CSRC, "lora_api.hip"), os.path.join(SAN, "host_check.cpp")):
        objs.append(str(tmp_path / (os.path.basename(src) + ".o")))
        res = subprocess.run([HIPCC, "-x", "hip", f"--offload-arch={B.ARCH}", "-O1", "-g", "-std=c++17", "-c",
                              f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"] + B.DEVICE_FLAGS + host_san +
                             [src, "-o", objs[-1]], capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-4000:]
    # the scheduler and the CPU LoRA kernel: plain C++
    for src in ("lora_sched.cpp", "lora_cpu.cpp"):
        objs.append(str(tmp_path / (src + ".o")))
        res = subprocess.run([CLANGXX, "-c", "-O1", "-g", "-std=c++17", f"-I{os.path.join(ROOT, 'include')}"] + san +
                             [os.path.join(CSRC, src), "-o", objs[-1]], capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-4000:]
    exe = str(tmp_path / "host_check")
    res = subprocess.run([CLANGXX] + san + objs + ["-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64",
                                                   "-o", exe], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, (run.stdout[-2000:], run.stderr[-6000:])
    assert "all checks passed" in run.stdout

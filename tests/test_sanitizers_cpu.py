"""AddressSanitizer + UndefinedBehaviorSanitizer runs of the host code (CPU).

The oracle is rebuilt with gcc under ASan/UBSan and its pin tests run
against that build; the host half of libtq (parser, planner, kernel source
generator, C ABI: program.cpp, jit.cpp, tq_abi.cpp) is rebuilt with the host
compilation under ASan/UBSan (device code unchanged, the kernels object of the
normal build linked in) and the C-ABI and planner tests run against it.  Each
run is a child process with the sanitizer runtime preloaded; any report ends
it with a non-zero status.  The sanitized libraries live in a temporary
directory and are never loaded by the product path.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2003_02989_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANGXX = "/opt/rocm/llvm/bin/clang++"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}

ORACLE_TESTS = ["test_oracle_gates.py", "test_oracle_closed_forms.py", "test_oracle_bruteforce.py",
                "test_oracle_gradients.py", "test_oracle_sampling.py", "test_oracle_sampled.py",
                "test_oracle_noise.py", "test_oracle_pauli_exp.py", "test_oracle_shift.py"]
HOST_TESTS = ["test_abi_cpu.py", "test_plan_cpu.py"]


def _gcc_runtime():
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _clang_runtime():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


def _run_tests(tests, env_extra, preload):
    env = dict(os.environ, **SAN_ENV, **env_extra, LD_PRELOAD=preload)
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"]
    cmd += [os.path.join(ROOT, "tests", t) for t in tests]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out


def test_oracle_under_asan_ubsan(tmp_path):
    rt = _gcc_runtime()
    if rt is None:
        pytest.skip("gcc's libasan is not installed")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer", "-o", lib, os.path.join(ROOT, "oracle", "tq_oracle.c"), "-lm"])
    _run_tests(ORACLE_TESTS, {"TQ_ORACLE_LIB": lib}, rt)


def test_host_runtime_under_asan_ubsan(tmp_path):
    rt = _clang_runtime()
    kobj = os.path.join(PKG, "_build", "kernels.hip.o")
    if rt is None or not os.path.exists(CLANGXX):
        pytest.skip("the ROCm clang ASan runtime is not installed")
    if not os.path.exists(kobj):
        pytest.skip("libtq is not built (python -m paper_2003_02989_amd.build)")
    # host compilation sanitized, device compilation as in the normal build
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "_build")]
    procs, objs = [], []
    for src in ("program.cpp", "tq_abi.cpp", "jit.cpp"):
        obj = str(tmp_path / (src + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC] + flags + ["-c", os.path.join(PKG, "csrc", src), "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
    for p in procs:
        out = p.communicate()[0]
        assert p.returncode == 0, out.decode()[-3000:]
    lib = str(tmp_path / "libtq_san.so")
    subprocess.check_call([CLANGXX, "-shared", "-fPIC", "-fsanitize=address,undefined", "-shared-libasan", "-o", lib]
                          + objs + [kobj, "-L/opt/rocm/lib", "-lamdhip64", "-lhiprtc", "-pthread",
                                    "-Wl,--no-undefined", "-Wl,-rpath,/opt/rocm/lib"])
    _run_tests(HOST_TESTS, {"TQ_LIB_PATH": lib}, rt)

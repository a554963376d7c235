"""AddressSanitizer and UndefinedBehaviorSanitizer builds (CPU only, no device code).

ROCm's clang builds everything here, so that one shared sanitizer runtime
serves every instrumented object; the library's host code is compiled with the
sanitizers on its host pass only (no device code is built).
  * tests/sanitize/oracle_driver.c with oracle/na_ref.c: every oracle entry
    point on small problems of each rank, including dilation, causal axes and
    windows as large as the extent; leaks are checked too;
  * tests/sanitize/host_driver.cpp with na_api.cpp: every public entry point
    through valid, invalid and empty problems, with launchers that check the
    geometry each kernel is handed and events that read a modelled clock (the
    tuner's choice is predicted and checked); out-of-range enum values come
    from tests/sanitize/c_caller.c, compiled as C;
  * the whole `-m "not gpu"` suite, run in a child process against sanitized
    builds of libna_ref.so and of libna.so's host code (its launchers report
    that no device is present), with the runtime preloaded into Python.
Any report ends the run with a non-zero status.
"""
import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2403_04690_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
LLVM = "/opt/rocm/llvm/bin"
CLANG, CLANGXX = os.path.join(LLVM, "clang"), os.path.join(LLVM, "clang++")

SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
# host pass only: the device pass of a HIP compile gets none of these
HOST_SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-sanitize-recover=all"]
HIP_HOST_ONLY = ["-x", "hip", "--offload-host-only", "-O1", "-g", "-std=c++17", "-fPIC",
                 "-fno-omit-frame-pointer", "-I", INCLUDE, "-I", CSRC]
RUN_ENV = {"ASAN_OPTIONS": "detect_leaks=1:halt_on_error=1",
           "LSAN_OPTIONS": "suppressions=" + os.path.join(SAN, "lsan.supp"),
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        pytest.fail(f"{' '.join(cmd)} failed ({res.returncode}):\n{res.stdout[-4000:]}\n"
                    f"{err[-4000:]}")
    return res


@pytest.fixture(scope="module")
def build(tmp_path_factory):
    hipcc = shutil.which("hipcc")
    if not (hipcc and os.path.exists(CLANG) and os.path.exists(CLANGXX)):
        pytest.skip("ROCm clang and hipcc are needed for the sanitizer builds")
    out = tmp_path_factory.mktemp("sanitize")
    o = lambda name: str(out / name)
    compiles = [
        [CLANG, "-x", "c", "-std=c11", "-O1", "-g", "-fPIC", "-fopenmp", "-Wall", "-Wextra",
         "-Werror"] + SAN_FLAGS + ["-c", os.path.join(ROOT, "oracle", "na_ref.c"), "-o",
                                   o("na_ref.o")],
        [CLANG, "-x", "c", "-std=c11", "-O1", "-g", "-Wall", "-Wextra", "-Werror"] + SAN_FLAGS +
        ["-c", os.path.join(SAN, "oracle_driver.c"), "-o", o("oracle_driver.o")],
        [CLANG, "-x", "c", "-std=c11", "-O1", "-g", "-Wall", "-Wextra", "-Werror", "-I",
         INCLUDE] + SAN_FLAGS + ["-c", os.path.join(SAN, "c_caller.c"), "-o", o("c_caller.o")],
        [hipcc] + HIP_HOST_ONLY + HOST_SAN_FLAGS +
        ["-c", os.path.join(CSRC, "na_api.cpp"), "-o", o("na_api.o")],
        [hipcc] + HIP_HOST_ONLY + HOST_SAN_FLAGS +
        ["-c", os.path.join(SAN, "host_driver.cpp"), "-o", o("host_driver.o")],
        [hipcc] + HIP_HOST_ONLY + HOST_SAN_FLAGS +
        ["-c", os.path.join(SAN, "no_device.cpp"), "-o", o("no_device.o")],
    ]
    with concurrent.futures.ThreadPoolExecutor(6) as ex:
        list(ex.map(_run, compiles))
    _run([CLANG] + SAN_FLAGS + ["-fopenmp", o("oracle_driver.o"), o("na_ref.o"), "-lm", "-o",
                                o("oracle_driver")])
    _run([CLANGXX] + SAN_FLAGS + [o("host_driver.o"), o("na_api.o"), o("c_caller.o"), "-o",
                                  o("host_driver")])
    # shared builds for the Python suite: the runtime comes from the preload
    _run([CLANG, "-shared", "-shared-libasan", "-fopenmp"] + SAN_FLAGS +
         [o("na_ref.o"), "-lm", "-o", o("libna_ref.so")])
    rocm_lib = os.path.realpath(os.path.join(LLVM, "..", "..", "..", "lib"))
    _run([CLANGXX, "-shared", "-shared-libasan"] + SAN_FLAGS +
         [o("na_api.o"), o("no_device.o"), "-L", rocm_lib, "-lamdhip64",
          f"-Wl,-rpath,{rocm_lib}", "-o", o("libna.so")])
    runtime = _run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"]).stdout.strip()
    assert os.path.isabs(runtime) and os.path.exists(runtime), runtime
    return out, runtime


def test_oracle_driver_is_clean(build):
    out, _ = build
    res = subprocess.run([str(out / "oracle_driver")], capture_output=True, text=True,
                         env={**os.environ, **RUN_ENV, "OMP_NUM_THREADS": "2"}, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip() == "ok oracle"


def test_host_driver_is_clean(build):
    out, _ = build
    res = subprocess.run([str(out / "host_driver")], capture_output=True, text=True,
                         env={**os.environ, **RUN_ENV}, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    words = res.stdout.split()
    assert words[:2] == ["ok", "host"], res.stdout
    assert int(words[2]) > 100000 and int(words[3]) > 1000  # checks, stubbed launches


def test_cpu_suite_under_sanitizers(build):
    out, runtime = build
    # reports go to files: pytest's capture of stderr would hide them when the
    # child ends on the first one
    report = str(out / "report")
    env = {**os.environ, **RUN_ENV, "LD_PRELOAD": runtime,
           # the interpreter and its extension modules keep memory until exit
           "ASAN_OPTIONS": f"detect_leaks=0:halt_on_error=1:log_path={report}",
           "UBSAN_OPTIONS": f"halt_on_error=1:print_stacktrace=1:log_path={report}",
           "NA_LIBRARY": str(out / "libna.so"), "NA_REF_LIBRARY": str(out / "libna_ref.so")}
    # the child maps the sanitized builds, not the regular ones
    probe = ("import oracle, paper_2403_04690_amd as na; oracle._load(); na.load_library(); "
             "print(''.join(l for l in open('/proc/self/maps') if 'libna' in l or 'asan' in l))")
    res = subprocess.run([sys.executable, "-c", probe], capture_output=True, text=True, env=env,
                         cwd=ROOT, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    for lib in (str(out / "libna.so"), str(out / "libna_ref.so"), runtime):
        assert os.path.realpath(lib) in res.stdout or lib in res.stdout, (lib, res.stdout)
    res = subprocess.run([sys.executable, "-m", "pytest", "tests", "-x", "-q", "-m", "not gpu",
                          "-p", "no:cacheprovider", "--ignore",
                          os.path.join("tests", "test_sanitizers.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=900)
    reports = "".join(open(f).read() for f in sorted(glob.glob(report + "*")))
    tail = (res.stdout + res.stderr)[-4000:] + reports[-6000:]
    assert res.returncode == 0 and not reports, tail
    assert "passed" in res.stdout and "failed" not in res.stdout, tail

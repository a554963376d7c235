"""Build paper_2403_04690_amd/libna.so (HIP kernels for gfx950 + the C ABI) with hipcc."""
import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libna.so")

SOURCES = ["na_fwd.hip", "na_bwd.hip", "na_unfused.hip", "na_debug.hip", "na_api.cpp"]
ARCH = os.environ.get("NA_OFFLOAD_ARCH", "gfx950")
# Packed fp32 instructions stay off: the compiler must not form v_pk_*_f32.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
         "-Werror=uninitialized", "-Werror=sometimes-uninitialized",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         # keep matrix-core results in ordinary VGPRs (no AGPR copies around the softmax)
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         # no NaN inputs are supported, so max() needs no NaN canonicalisation
         # (infinities stay honoured: masked scores are -inf)
         "-fno-honor-nans",
         "-I", INCLUDE, "-I", CSRC]


def _compile(src, verbose, extra=()):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = ["hipcc"] + FLAGS + list(extra) + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip() and verbose:
        print(err, flush=True)
    return obj


def build_pyext(verbose=False):
    """Compile the binding's optional argument-marshalling extension (_na_fast, host C only)."""
    import sysconfig

    out = os.path.join(PKG, "_na_fast" + sysconfig.get_config_var("EXT_SUFFIX"))
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror",
           "-I", sysconfig.get_paths()["include"], "-I", INCLUDE,
           os.path.join(CSRC, "na_pyext.c"), "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def build(verbose=False, jobs=None, out=None, extra_flags=()):
    """Compile every source and link libna.so (or `out`); extra_flags go to every hipcc call."""
    global BUILD
    build_dir = BUILD if out is None else os.path.join(os.path.dirname(out), "_build")
    os.makedirs(build_dir, exist_ok=True)
    saved, BUILD = BUILD, build_dir
    try:
        return _build(verbose, jobs, out or LIB, list(extra_flags))
    finally:
        BUILD = saved


def _build(verbose, jobs, lib, extra):
    jobs = jobs or min(len(SOURCES), max(1, os.cpu_count() or 1), 16)
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, extra), SOURCES))
    tmp = lib + ".tmp"
    cmd = ["hipcc", "-shared", "-fPIC", f"--offload-arch={ARCH}"] + objs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    build_pyext(verbose="-v" in sys.argv)

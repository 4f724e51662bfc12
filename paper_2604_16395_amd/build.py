"""Build libs2l.so (HIP kernels for gfx950 + the C-ABI layer) in place.

Usage: python -m paper_2604_16395_amd.build [-v] [--sanitize]

--sanitize also builds _build/san/libs2l.so: the same device objects, with the host C++
(argument validation, the host planner, the scheduler) compiled by g++ under AddressSanitizer
and UndefinedBehaviorSanitizer.  Load it with S2L_LIBRARY=<path> and the ASan runtime first in
LD_PRELOAD (tests/test_sanitize_cpu.py runs the host-side test files that way); it is for the
CPU tests, not for GPU runs.
"""
import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libs2l.so")
ARCH = "gfx950"


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


COMMON = ["-O3", "-fPIC", "-std=c++17", "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-result"]
# No packed fp32 ops in device code (v_pk_*_f32 are avoided on this hardware).
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-munsafe-fp-atomics"]


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    jobs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        jobs.append([hipcc, "-x", "hip", *COMMON, *DEVICE, "-c", src, "-o", obj])
    for src in sorted(glob.glob(os.path.join(CSRC, "*.cpp"))):
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        jobs.append([hipcc, *COMMON, "-c", src, "-o", obj])

    def run(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        p = subprocess.run(cmd, capture_output=True, text=True)
        out = "\n".join(l for l in (p.stdout + p.stderr).splitlines()
                        if "packed-fp32-ops" not in l and l.strip())
        if p.returncode != 0:
            raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{out}")
        if verbose and out:
            print(out)
        return cmd[-1]

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        objs = list(ex.map(run, jobs))
    tmp = LIB + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    run(cmd)
    os.replace(tmp, LIB)
    return LIB


SAN = os.path.join(BUILD, "san")
SAN_LIB = os.path.join(SAN, "libs2l.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def build_sanitized(verbose=False):
    """Host sources under ASan + UBSan (g++), linked with the device objects of build()."""
    build(verbose)
    os.makedirs(SAN, exist_ok=True)
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(_hipcc())))
    gxx = os.environ.get("CXX") or shutil.which("g++")
    if not gxx:
        raise RuntimeError("g++ not found")
    objs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "*.cpp"))):
        obj = os.path.join(SAN, os.path.basename(src) + ".o")
        cmd = [gxx, "-std=c++17", "-O1", "-g", "-fPIC", *SAN_FLAGS, "-D__HIP_PLATFORM_AMD__",
               "-I", os.path.join(rocm, "include"), "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    dev = sorted(glob.glob(os.path.join(BUILD, "*.hip.o")))
    lib_dir = os.path.join(rocm, "lib")
    cmd = [gxx, "-shared", *SAN_FLAGS, "-o", SAN_LIB, *dev, *objs, "-L", lib_dir, "-lamdhip64",
           f"-Wl,-rpath,{lib_dir}"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return SAN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    if "--sanitize" in sys.argv:
        print(build_sanitized(verbose="-v" in sys.argv))

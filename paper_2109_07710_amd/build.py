"""Build libconvbwd.so (the HIP kernels and the C-ABI) for gfx950, in-tree.

    python -m paper_2109_07710_amd.build

Every source is compiled by hipcc for gfx950 only, with packed fp32
instructions disabled, and linked into paper_2109_07710_amd/libconvbwd.so;
the benchmark's peak-measurement kernels go into libcbwpeaks.so.
"""
import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libconvbwd.so")
# measured machine ceilings for the benchmark's roofline (include/cbw_peaks.h)
PEAKS_LIB = os.path.join(HERE, "libcbwpeaks.so")
PEAKS_SOURCES = ["peaks.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["api.cpp", "plan.cpp", "bwd_data.hip", "bwd_data_rows.hip", "bwd_data_pw.hip", "bwd_weight.hip", "mask_kernels.hip", "elementwise.hip", "layout.hip"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result"]
DEVICE = ["-x", "hip", "--offload-arch=gfx950",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src, verbose):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + COMMON
    if src != "plan.cpp":  # plan.cpp is plain host C++
        cmd += DEVICE
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s" % (src, err))
    if verbose and err.strip():
        print(err)
    return obj


def _link(objs, lib, verbose):
    tmp = lib + ".tmp"
    # -z defs: a symbol missing from the objects fails the link here rather
    # than the library's load on the device host
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-Wl,-z,defs", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed (%s)\n%s" % (os.path.basename(lib), r.stderr))
    os.replace(tmp, lib)


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + PEAKS_SOURCES
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        objs = dict(zip(srcs, ex.map(lambda s: _compile(s, verbose), srcs)))
    _link([objs[s] for s in SOURCES], LIB, verbose)
    _link([objs[s] for s in PEAKS_SOURCES], PEAKS_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

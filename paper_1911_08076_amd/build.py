"""Build libifq.so (HIP for gfx950 + host C++) into this package directory.

Usage: python paper_1911_08076_amd/build.py (runs without importing the
package, which needs the library to exist)
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libifq.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["ifq_api.cpp", "ifq_conv.hip", "ifq_conv_mfma.hip", "ifq_conv_halo.hip", "ifq_conv_w2.hip", "ifq_conv_wp.hip", "ifq_noalloc.hip",
           "ifq_conv_small.hip", "ifq_pool.hip", "ifq_thresholds.hip"]


def build(verbose=False):
    """Compile every source to an object in parallel, then link libifq.so."""
    from concurrent.futures import ThreadPoolExecutor
    flags = [HIPCC, "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
             "-fvisibility=hidden", "-ffp-contract=off",
             # no packed-fp32 instructions anywhere in device code
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", INCLUDE, "-I", CSRC]
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    tag = "%d" % os.getpid()

    def compile_one(src):
        obj = os.path.join(objdir, os.path.splitext(src)[0] + "." + tag + ".o")
        cmd = flags + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        return obj, r

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        results = list(ex.map(compile_one, SOURCES))
    objs = []
    for obj, r in results:
        err = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                        if "packed-fp32-ops" not in l)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + err)
        objs.append(obj)
    tmp = LIB + ".tmp" + tag
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-Wl,--no-undefined",
           "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    for o in objs:
        os.remove(o)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv))

"""Build ``libzpp.so`` (the HIP kernels and the C ABI) for gfx950 in-tree.

    python -m paper_2407_01614_amd.build          # builds paper_2407_01614_amd/libzpp.so
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libzpp.so")
# the plain HBM streams that bench.py times beside the kernels (not the path)
CEILING_LIB = os.path.join(PKG, "libzpp_ceiling.so")
CEILING_SOURCES = ["ceiling.hip"]

SOURCES = ["zpp_api.hip", "adam.hip", "refresh.hip", "quant.hip", "gather.hip", "fused.hip",
           "qgz.hip", "receive_adam.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-fvisibility=hidden",
    "-Wall",
    "-Werror",
    # IEEE fp32 division and square root, denormals kept: the quantization
    # codes and scales must be the correctly rounded binary32 results.
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero",
    "-fno-fast-math",
    # no packed-fp32 VALU forms (v_pk_{add,mul,fma}_f32) in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    for cand in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), "hipcc"):
        if os.path.sep not in cand or os.path.exists(cand):
            return cand
    return "hipcc"


def build(out=LIB, defines=(), verbose=False, sources=SOURCES):
    """Compile the HIP sources of the path into one shared library."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, *["-D" + d for d in defines], "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in sources], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so; that
    # warning is expected, anything else is shown
    noise = "not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l and l.strip())
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stderr)
    if err and verbose:
        print(err, file=sys.stderr)
    os.replace(tmp, out)
    return out


def build_ceiling(verbose=False):
    """Compile the measurement streams into libzpp_ceiling.so."""
    return build(out=CEILING_LIB, verbose=verbose, sources=CEILING_SOURCES)


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_ceiling(verbose=True))

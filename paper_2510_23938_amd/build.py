"""Builds ``libhv.so`` (the HIP kernels and the C ABI) for gfx950 with hipcc, in-tree."""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
_ROOT = os.path.dirname(_HERE)
CSRC = os.path.join(_HERE, "csrc")
OUT = os.path.join(_HERE, "libhv.so")
BUILD_DIR = os.path.join(_HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # no packed-FP32 instruction selection anywhere in this library.  The
    # feature is a device (gfx950) one, but clang forwards no -cc1 option
    # through -Xarch_device, so both passes get it and the x86 host pass
    # prints that it does not know the feature; that notice is dropped below.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(_ROOT, "include"), "-I", CSRC,
]
_HOST_PASS_NOTICE = "'-packed-fp32-ops' is not a recognized feature for this target (ignoring feature)"


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    r = subprocess.run([HIPCC, *FLAGS, "-x", "hip", "-c", src, "-o", obj], capture_output=True, text=True)
    rest = "".join(ln for ln in r.stderr.splitlines(keepends=True) if _HOST_PASS_NOTICE not in ln)
    if rest:
        print(rest, end="", file=sys.stderr)
    if r.returncode != 0:
        raise subprocess.CalledProcessError(r.returncode, r.args, r.stdout, r.stderr)
    return obj


def build() -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = OUT + ".tmp"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], check=True)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build())

"""Builds the host checks in tests/host_checks/_build: a copy of libhv whose
host code is compiled with AddressSanitizer and UndefinedBehaviorSanitizer
(the device code is compiled as usual; the sanitizers go to the host side
only, through -Xarch_host), and host_checks.c linked against it with the same
sanitizers.  The product library is not touched."""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2510_23938_amd", "csrc")
OUT = os.path.join(HERE, "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
LIB = os.path.join(OUT, "libhv_sanitized.so")
EXE = os.path.join(OUT, "host_checks")

# host side only: each sanitizer flag right after -Xarch_host
HOST_SANITIZERS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                   "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC, *HOST_SANITIZERS]


def _compile(src: str) -> str:
    obj = os.path.join(OUT, os.path.basename(src) + ".o")
    subprocess.run([HIPCC, *FLAGS, "-x", "hip", "-c", src, "-o", obj], check=True)
    return obj


def build() -> str:
    os.makedirs(OUT, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", LIB, *HOST_SANITIZERS],
                   check=True)
    # the driver is plain C on the host: the C compiler of the same toolchain, so one sanitizer runtime
    subprocess.run([CLANG, "-std=c11", "-O1", "-g", "-Wall", "-Wextra", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
                    os.path.join(HERE, "host_checks.c"), "-o", EXE, LIB,
                    "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
                    f"-Wl,-rpath,{OUT}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"], check=True)
    return EXE


if __name__ == "__main__":
    print(build(), file=sys.stderr)

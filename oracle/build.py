"""Builds the CPU oracle (``liboracle.so``) with the host C compiler.

Test infrastructure: compiled so the checker exists; the product library never
links or loads it.
"""
import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))


def build() -> str:
    src = os.path.join(_HERE, "hv_oracle.c")
    out = os.path.join(_HERE, "liboracle.so")
    tmp = out + ".tmp"
    subprocess.run(
        ["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared", "-pthread", src, "-o", tmp],
        check=True,
    )
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())

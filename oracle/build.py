"""Builds the oracle's shared library (test infrastructure; see oracle/__init__.py)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def build() -> str:
    src = os.path.join(HERE, "oracle.cpp")
    out = os.path.join(HERE, "liboracle.so")
    tmp = out + ".tmp"
    subprocess.run(["g++", "-O2", "-std=c++17", "-Wall", "-Wextra", "-shared", "-fPIC",
                    "-o", tmp, src], check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())

"""Build and run the microbenchmarks on one MI355X (gfx950).

    python microbench/run.py            # builds microbench/_build/msda_micro, runs it, prints the table

The binary is built with the same hipcc flags as the library. It allocates about 0.3 GB of device
memory and runs for a few seconds.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
BUILD = os.path.join(HERE, "_build")
SRC = os.path.join(HERE, "msda_micro.hip")
EXE = os.path.join(BUILD, "msda_micro")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-munsafe-fp-atomics"]


def build() -> str:
    os.makedirs(BUILD, exist_ok=True)
    subprocess.run([os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")] + FLAGS + ["-o", EXE, SRC], check=True)
    return EXE


if __name__ == "__main__":
    if "--no-build" not in sys.argv or not os.path.exists(EXE):
        build()
    if "--build-only" not in sys.argv:
        sys.exit(subprocess.run([EXE]).returncode)

"""Compile synth/rspec_fast.c into synth/_rspec_fast.so with gcc -fopenmp."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SO = os.path.join(HERE, "_rspec_fast.so")


def build() -> str:
    src = os.path.join(HERE, "rspec_fast.c")
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off", src, "-o", SO + ".tmp"],
                   check=True)
    os.replace(SO + ".tmp", SO)
    return SO


if __name__ == "__main__":
    print(build())

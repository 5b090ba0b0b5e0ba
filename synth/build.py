"""Build the two generator libraries in-tree (host: gcc + OpenMP; device: hipcc for gfx950)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + r.stdout + r.stderr)


def build(verbose: bool = False) -> None:
    src = os.path.join(HERE, "csrc")
    _run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared", "-std=c11",
          os.path.join(src, "synth_host.c"), "-o", os.path.join(HERE, "libsynth_host.so"), "-lm"])
    _run([HIPCC, "--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
          "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          os.path.join(src, "synth_device.hip"), "-o", os.path.join(HERE, "libsynth_device.so")])
    if verbose:
        print("built synth libraries")


if __name__ == "__main__":
    build(verbose=True)

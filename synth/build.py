"""Builds synth/libsynth.so (host + gfx950 device code) with hipcc."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libsynth.so")

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", "--offload-arch=gfx950", "-fopenmp",
    # host and device must round identically: no contraction of a*b+c into fma
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


SAN_LIB = os.path.join(HERE, "libsynth_san.so")
# host code only: each sanitizer flag applies to the host compilation (device code is unchanged)
SAN_FLAGS = ["-O1", "-g", "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-shared-libsan"]


def build(verbose=False, sanitize=False):
    """sanitize: a separate libsynth_san.so whose host code carries AddressSanitizer and
    UndefinedBehaviorSanitizer, loaded instead of libsynth.so when MPC_SANITIZE=1."""
    src = os.path.join(HERE, "synth.hip")
    out = SAN_LIB if sanitize else LIB
    cmd = ["hipcc", *FLAGS, *(SAN_FLAGS if sanitize else []), src, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True, stderr=None if verbose else subprocess.DEVNULL)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    import sys
    print(build(verbose=True, sanitize="--sanitize" in sys.argv))

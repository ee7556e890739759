"""Builds oracle/liboracle.so (plain C++17, fp64) with the host compiler. Test infrastructure."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


SAN_LIB = os.path.join(HERE, "liboracle_san.so")
CLANG = "/opt/rocm/lib/llvm/bin/clang++"


def build(verbose=False, sanitize=False):
    """sanitize: a separate liboracle_san.so built by clang with AddressSanitizer and
    UndefinedBehaviorSanitizer (the runtime the synth library's sanitized build uses too), loaded
    instead of liboracle.so when MPC_SANITIZE=1 (see tests/sanitize.sh)."""
    src = os.path.join(HERE, "mpcache_oracle.cpp")
    out = SAN_LIB if sanitize else LIB
    if sanitize:
        cmd = [CLANG, "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
               "-shared-libsan", "-Wall", "-Wextra", src, "-o", out + ".tmp"]
    else:
        cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-Wall", "-Wextra", src, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    import sys
    print(build(verbose=True, sanitize="--sanitize" in sys.argv))

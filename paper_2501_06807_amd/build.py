"""Builds paper_2501_06807_amd/libmpcache.so from csrc/*.hip for gfx950 with hipcc, and the
read-ceiling measurement kernel (libmpc_ceiling.so, used by the bench only)."""
import concurrent.futures as cf
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libmpcache.so")
CEILING_LIB = os.path.join(HERE, "libmpc_ceiling.so")
BUILD_DIR = os.path.join(ROOT, "_build", "mpcache")

CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))


def build(verbose=False):
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))
    objs = [os.path.join(BUILD_DIR, os.path.basename(s) + ".o") for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        futs = [ex.submit(_run, ["hipcc", *CFLAGS, "-c", s, "-o", o], verbose) for s, o in zip(srcs, objs)]
        for f in futs:
            f.result()
    _run(["hipcc", "-shared", "--offload-arch=gfx950", *objs, "-o", LIB + ".tmp"], verbose)
    os.replace(LIB + ".tmp", LIB)
    _run(["hipcc", *CFLAGS, "-shared", os.path.join(HERE, "ceiling", "read_ceiling.hip"), "-o", CEILING_LIB + ".tmp"],
         verbose)
    os.replace(CEILING_LIB + ".tmp", CEILING_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

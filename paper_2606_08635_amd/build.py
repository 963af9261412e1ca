"""Builds ``libskv.so`` (the C-ABI codec library) for gfx950 with hipcc.

Every source is compiled with contraction off (so ``x * r + c`` is never fused
and each binary32 operation rounds once), correctly rounded binary32 division,
and packed-fp32 instructions disabled.
"""
import concurrent.futures
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libskv.so")
# streaming reference kernels (measurement only), a library of their own
CEILING_LIB = os.path.join(HERE, "libskv_ceiling.so")
CEILING_SOURCES = ["ceiling.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["skv_api.cpp", "score.hip", "attn.hip", "select.hip", "pack.hip", "unpack.hip", "upgrade.hip", "groups.hip",
           "link.hip"]
FLAGS = [
    "-x", "hip", "-std=c++17", "-O3", "--offload-arch=gfx950", "-fPIC",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument", "-I", INCLUDE,
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stdout}\n{res.stderr}")
    noise = "packed-fp32-ops"  # the host pass does not know the device-only feature
    for line in res.stderr.splitlines():
        if line.strip() and noise not in line and verbose:
            print(line)
    return obj


def _link(objs, lib: str, verbose: bool) -> None:
    tmp = lib + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)


def build(verbose: bool = False, jobs: int = 6) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES + CEILING_SOURCES))
    _link(objs[:len(SOURCES)], LIB, verbose)
    _link(objs[len(SOURCES):], CEILING_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

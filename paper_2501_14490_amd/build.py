"""Build ``libmfpsn.so`` (gfx950) from ``csrc/`` with hipcc.

The kernel source is compiled once per storage type and range of orders k so
the (large, fully unrolled) instantiations build in parallel, then linked
with the C-ABI layer into ``paper_2501_14490_amd/libmfpsn.so``.

    python -m paper_2501_14490_amd.build [--jobs N] [--force]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmfpsn.so")
ARCH = "gfx950"

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

# Device code: IEEE single precision with denormals, no FMA contraction (the
# float sums are pinned to a sequential order), packed-FP32 instructions off.
DEVICE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC", "-ffp-contract=off",
    "-fno-gpu-flush-denormals-to-zero", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
HOST_FLAGS = ["-O2", "-std=c++20", "-fPIC", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I/opt/rocm/include"]

K_RANGES = [(1, 8), (9, 12), (13, 16), (17, 20), (21, 23), (24, 26), (27, 29), (30, 31), (32, 32)]
DTYPES = [0, 1, 2]  # f32, bf16, q8.8


def _units():
    """(object, compile command, sources it depends on) of every translation unit."""
    src = os.path.join(CSRC, "mfpsn_kernels.hip")
    # the headers the kernel source includes (not the public header: the
    # kernels see only the internal interface)
    headers = [os.path.join(CSRC, "mfpsn_internal.h"), os.path.join(CSRC, "mfpsn_surrogate.h")]
    api_headers = [*headers, os.path.join(INCLUDE, "mfpsn.h")]
    units = []
    for dt in DTYPES:
        for lo, hi in K_RANGES:
            obj = os.path.join(BUILD, f"kernels_d{dt}_k{lo}-{hi}.o")
            units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}",
                                f"-DMFPSN_TU_DTYPE={dt}", f"-DMFPSN_TU_KLO={lo}",
                                f"-DMFPSN_TU_KHI={hi}", "-c", src, "-o", obj], [src, *headers]))
    bn_src = os.path.join(CSRC, "mfpsn_bn.hip")
    obj = os.path.join(BUILD, "bn.o")
    units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", bn_src, "-o", obj],
                  [bn_src, os.path.join(CSRC, "mfpsn_bn.h"), os.path.join(INCLUDE, "mfpsn.h")]))
    qg_src = os.path.join(CSRC, "mfpsn_qgrad.hip")
    obj = os.path.join(BUILD, "qgrad.o")
    units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", qg_src, "-o", obj],
                  [qg_src, os.path.join(CSRC, "mfpsn_qgrad.h")]))
    tl_src = os.path.join(CSRC, "mfpsn_tl.hip")
    tl_deps = [tl_src, os.path.join(CSRC, "mfpsn_tl.h"), os.path.join(CSRC, "mfpsn_surrogate.h"),
               os.path.join(INCLUDE, "mfpsn.h")]
    for tag, flag in (("d0", "-DMFPSN_TL_DTYPE=0"), ("d1", "-DMFPSN_TL_DTYPE=1"), ("d2", "-DMFPSN_TL_DTYPE=2"),
                      ("dispatch", None)):
        obj = os.path.join(BUILD, f"tl_{tag}.o")
        units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", *([flag] if flag else []),
                            "-c", tl_src, "-o", obj], tl_deps))
    chain_src = os.path.join(CSRC, "mfpsn_chain.hip")
    obj = os.path.join(BUILD, "chain.o")
    units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", chain_src, "-o", obj],
                  [chain_src, os.path.join(CSRC, "mfpsn_chain.h"), os.path.join(INCLUDE, "mfpsn.h")]))
    stream_src = os.path.join(CSRC, "mfpsn_stream.hip")
    obj = os.path.join(BUILD, "stream.o")
    units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", stream_src, "-o", obj],
                  [stream_src, os.path.join(CSRC, "mfpsn_stream.h"), *api_headers]))
    na_src = os.path.join(CSRC, "mfpsn_noalloc.hip")
    obj = os.path.join(BUILD, "noalloc.o")
    units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", na_src, "-o", obj],
                  [na_src, os.path.join(INCLUDE, "mfpsn.h")]))
    obj = os.path.join(BUILD, "kernels_misc.o")
    units.append((obj, [HIPCC, *DEVICE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-DMFPSN_TU_MISC",
                        "-c", src, "-o", obj], [src, *headers]))
    for name in ("mfpsn_api.cpp", "mfpsn_api_ext.cpp", "mfpsn_dispatch.cpp"):
        obj = os.path.join(BUILD, name.replace(".cpp", ".o"))
        cpp = os.path.join(CSRC, name)
        units.append((obj, ["g++", *HOST_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", cpp, "-o", obj],
                      [cpp, os.path.join(CSRC, "mfpsn_stream.h"), os.path.join(CSRC, "mfpsn_qgrad.h"),
                       os.path.join(CSRC, "mfpsn_bn.h"), os.path.join(CSRC, "mfpsn_validate.h"),
                       os.path.join(CSRC, "mfpsn_chain.h"), os.path.join(CSRC, "mfpsn_tl.h"), *api_headers]))
    return units


def build(jobs: int | None = None, force: bool = True, verbose: bool = False) -> str:
    """Compile every translation unit and link libmfpsn.so; returns its path.
    With force=False, units whose object is newer than every source it
    depends on are kept."""
    os.makedirs(BUILD, exist_ok=True)
    todo = []
    for obj, cmd, deps in _units():
        newest = max(os.path.getmtime(p) for p in deps)
        if force or not os.path.exists(obj) or os.path.getmtime(obj) < newest:
            todo.append((obj, cmd))
    jobs = jobs or min(8, os.cpu_count() or 1)
    t0 = time.time()

    def run(item):
        obj, cmd = item
        t = time.time()
        p = subprocess.run(cmd, capture_output=True, text=True)
        out = "\n".join(l for l in (p.stdout + p.stderr).splitlines()
                        if "packed-fp32-ops" not in l)
        if p.returncode != 0:
            raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{out}")
        if verbose:
            print(f"  built {os.path.basename(obj)} in {time.time() - t:.1f}s", flush=True)
        return obj

    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(run, todo))
    objs = [obj for obj, _, _ in _units()]
    tmp = LIB + f".tmp{os.getpid()}"
    link = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    p = subprocess.run(link, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(link)}\n{p.stdout}{p.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"libmfpsn.so linked ({len(todo)} units compiled, {time.time() - t0:.1f}s)", flush=True)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--force", action="store_true")
    args = ap.parse_args(argv)
    build(args.jobs, force=args.force, verbose=True)


if __name__ == "__main__":
    sys.exit(main())

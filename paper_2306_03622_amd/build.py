"""Builds libtorpor.so (HIP, gfx950) in-tree, plus the host-only planning library.

    python -m paper_2306_03622_amd.build [--jobs N] [--sanitize]

``libtorpor.so`` holds the C ABI of include/torpor.h and include/torpor_plan.h with all
kernels; ``libtorpor_probe.so`` the peak probes of include/torpor_probe.h that the
benchmark measures its rooflines against. ``libtorpor_host.so`` is the same host-side bookkeeping (validation, chunk
plan, arena) compiled with g++ alone, optionally with ASan/UBSan, for host-only tests.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libtorpor.so")
HOST_LIB = os.path.join(PKG, "libtorpor_host.so")
PROBE_LIB = os.path.join(PKG, "libtorpor_probe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

CORE = ["core/model.cpp", "core/arena.cpp", "core/partition.cpp", "core/sched.cpp", "core/plan_api.cpp", "core/errors.cpp"]
HIP_HOST = ["hip/runtime.cpp", "hip/executors.cpp", "hip/trace.cpp"]
PROBE = ["probe/peaks.hip"]
KERNELS = ["hip/scratch.hip", "kernels/gemm_bf16.hip", "kernels/gemv_bf16.hip", "kernels/linear_f32.hip", "kernels/norm.hip", "kernels/attention.hip",
           "kernels/pool_copy.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", f"-I{os.path.join(ROOT, 'include')}"]
# host translation units that use the HIP runtime API only
HOST_HIP = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]
# device code: gfx950 only; packed-fp32 instructions disabled; MFMA accumulators in ordinary
# VGPRs (the default accumulation-register form made the register allocator shuffle
# accumulators between register files inside the GEMM and attention loops: ~2,400 and ~700
# extra moves per instantiation set; the matrix-core probe ran at half rate because of it)
DEVICE = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-mllvm", "-amdgpu-mfma-vgpr-form"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{err}")
    return err


def _obj(src):
    return os.path.join(OUT, src.replace("/", "_").rsplit(".", 1)[0] + ".o")


def build(jobs: int = 8, sanitize: bool = False, verbose: bool = False) -> str:
    os.makedirs(OUT, exist_ok=True)
    cmds = []
    for src in CORE + HIP_HOST:
        cmds.append([HIPCC, *COMMON, *HOST_HIP, "-x", "c++", "-c", os.path.join(CSRC, src), "-o", _obj(src)])
    for src in KERNELS + PROBE:
        cmds.append([HIPCC, *COMMON, *DEVICE, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", _obj(src)])
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for msg in ex.map(_run, cmds):
            if verbose and msg:
                print(msg, file=sys.stderr)
    objs = [_obj(s) for s in CORE + HIP_HOST + KERNELS]
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", *DEVICE, "-o", tmp, *objs, "-lpthread"])
    os.replace(tmp, LIB)
    # peak probes of the benchmark (a library of their own, no part of the serving path)
    ptmp = PROBE_LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", *DEVICE, "-o", ptmp, *[_obj(s) for s in PROBE]])
    os.replace(ptmp, PROBE_LIB)
    build_host(HOST_LIB, sanitize)
    return LIB


# AddressSanitizer and UndefinedBehaviorSanitizer, every report fatal
SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def build_host(path: str = HOST_LIB, sanitize: bool = False) -> str:
    """The host-only planning library (g++ alone, no HIP), optionally under the sanitizers."""
    tmp = path + ".tmp"
    _run(["g++", "-O1" if sanitize else "-O2", "-std=c++17", "-fPIC", "-shared", "-fvisibility=hidden",
          *(SANITIZE if sanitize else []), f"-I{os.path.join(ROOT, 'include')}",
          *[os.path.join(CSRC, s) for s in CORE], "-o", tmp])
    os.replace(tmp, path)
    return path


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=8)
    ap.add_argument("--sanitize", action="store_true")
    ap.add_argument("-v", "--verbose", action="store_true")
    a = ap.parse_args()
    print(build(a.jobs, a.sanitize, a.verbose))

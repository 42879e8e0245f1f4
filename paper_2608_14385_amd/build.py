"""Build libdeamoe.so (HIP, gfx950) in-tree with hipcc, and the benchmark's
read-bandwidth probe libdeamoe_probe.so.

    python -m paper_2608_14385_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdeamoe.so")
SOURCES = ("api.hip", "route.hip", "gemm.hip", "combine.hip", "chain.hip", "small.hip")
PROBE_SRC = os.path.join(CSRC, "probe", "read_probe.hip")
PROBE_LIB = os.path.join(HERE, "libdeamoe_probe.so")

# Packed fp32 instructions are disabled for all device code.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src).replace(".hip", ".o"))
    cmd = [_hipcc(), *HIPCC_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if noise not in ln]
    if r.returncode:
        raise RuntimeError(f"hipcc failed on {src}:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(tmp, LIB)
    probe = _compile(PROBE_SRC, verbose)
    cmd = [_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", PROBE_LIB + ".tmp", probe]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(PROBE_LIB + ".tmp", PROBE_LIB)
    return LIB


# Host-side sanitizer flags for the C-ABI translation unit (device code is
# built as usual): AddressSanitizer and UndefinedBehaviorSanitizer, aborting
# on the first finding.
SAN_HOST_FLAGS = ("-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
                  "-Xarch_host -fno-sanitize-recover=undefined "
                  "-Xarch_host -fno-omit-frame-pointer").split()


def build_host_sanitized(out_dir: str, verbose: bool = False) -> str:
    """libdeamoe.so in out_dir with the host code of api.hip (validation,
    workspace layout, launch sequence) built under ASan and UBSan, linked
    with the regular objects of the kernel sources.  A process loading it
    needs clang's ASan runtime preloaded (asan_runtime())."""
    kernel_objs = [os.path.join(BUILD, s.replace(".hip", ".o")) for s in SOURCES if s != "api.hip"]
    if not all(os.path.exists(o) for o in kernel_objs):
        build(verbose)
    os.makedirs(out_dir, exist_ok=True)
    obj = os.path.join(out_dir, "api_san.o")
    cmd = [_hipcc(), *HIPCC_FLAGS, *SAN_HOST_FLAGS, "-g", "-c", os.path.join(CSRC, "api.hip"),
           "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError("hipcc failed on api.hip (sanitized):\n" + r.stdout + r.stderr)
    objs = [obj] + kernel_objs
    lib = os.path.join(out_dir, "libdeamoe.so")
    cmd = [_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *SAN_HOST_FLAGS[:4],
           "-shared-libasan", "-o", lib, *objs]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    return lib


def asan_runtime() -> str:
    """Path of clang's shared AddressSanitizer runtime (for LD_PRELOAD)."""
    return subprocess.run([_hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], check=True,
                          capture_output=True, text=True).stdout.strip()


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

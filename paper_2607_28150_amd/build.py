"""Build step for libsmartgen.so (gfx950 only): ``python -m paper_2607_28150_amd.build``.

Every ``csrc/*.hip`` file is compiled to an object with hipcc for gfx950 and
the objects are linked into ``libsmartgen.so`` next to this file.  Packed FP32
instruction selection is switched off for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
_ROOT = os.path.dirname(_HERE)
LIB_PATH = os.path.join(_HERE, "libsmartgen.so")
ARCH = "gfx950"

CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(_ROOT, "include"),
]

# Per-file additions.  topshare.hip: its histogram kernels hold 130 KB of LDS,
# so one workgroup per CU and a register budget above 256, where the compiler
# would put the MFMA accumulators in AGPRs and copy every value out before the
# vector work; the VGPR form fits the bf16 kernels in 256 VGPRs without spills.
FILE_FLAGS = {
    "topshare.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def _hipcc() -> str:
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _compile(src: str, obj: str, verbose: bool) -> None:
    cmd = [_hipcc(), *CFLAGS, *FILE_FLAGS.get(os.path.basename(src), []), "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so: harmless
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip() and verbose:
        print(err)


def build(verbose: bool = False, jobs: int = 8) -> str:
    srcs = sorted(glob.glob(os.path.join(_HERE, "csrc", "*.hip")))
    bdir = os.path.join(_ROOT, "_build")
    os.makedirs(bdir, exist_ok=True)
    objs = [os.path.join(bdir, os.path.basename(s)[:-4] + ".o") for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(lambda so: _compile(so[0], so[1], verbose), zip(srcs, objs)))
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def build_host_sanitized(out_path: str, jobs: int = 8) -> str:
    """The library with its host code (argument checks, dispatch) built with
    AddressSanitizer and UndefinedBehaviorSanitizer (device code unoptimised:
    the sanitized library is for CPU-only checks of the host side).  Load it with the
    clang ASan runtime preloaded."""
    srcs = sorted(glob.glob(os.path.join(_HERE, "csrc", "*.hip")))
    bdir = os.path.join(os.path.dirname(os.path.abspath(out_path)), "objs")
    os.makedirs(bdir, exist_ok=True)
    objs = [os.path.join(bdir, os.path.basename(s)[:-4] + ".o") for s in srcs]
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = ["-Xarch_host", "-O1", "-Xarch_host", "-g", "-Xarch_device", "-O0", "-std=c++17", "-fPIC",
             f"--offload-arch={ARCH}", *san,
             "-I", os.path.join(_ROOT, "include")]

    def one(so):
        r = subprocess.run([_hipcc(), *flags, "-c", so[0], "-o", so[1]], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (host, sanitized) failed for {so[0]}:\n{r.stderr}")

    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(one, zip(srcs, objs)))
    subprocess.run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *san, *objs, "-o", out_path], check=True,
                   capture_output=True)
    return out_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

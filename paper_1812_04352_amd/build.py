"""Build the HIP library liblp.so for gfx950 in-tree (hipcc, no JIT cache).

Every translation unit is compiled for gfx950 only, with packed-fp32 VALU
instructions disabled, then linked into paper_1812_04352_amd/liblp.so next to
this file. Objects go to paper_1812_04352_amd/_build/.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "liblp.so")
OBJ = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["lp_host.cpp", "lp_common.hip", "lp_loss.hip", "lp_dense_f32.hip", "lp_dense_f64.hip",
           "lp_dense_mfma.hip", "lp_dense_wide.hip", "lp_conv.hip", "lp_noalloc.hip"]

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    "-Wno-unused-result",
]


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


# Host-code sanitizers (AddressSanitizer, UndefinedBehaviorSanitizer) for the
# CPU-side checks: every flag goes to the host compilation only (-Xarch_host), the
# GPU code objects are the ordinary ones.
SAN_FLAGS = ["-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xarch_host", "-shared-libasan"]
SAN_SOURCES = ["lp_host.cpp", "lp_noalloc.hip"]  # the translation units with host logic beyond launches
SAN_OUT = os.path.join(OBJ, "liblp_san.so")


def sanitizer_runtime() -> str:
    """Path of the shared AddressSanitizer runtime (to be preloaded into a host
    process that is not itself instrumented, e.g. python)."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()


def build_sanitized(verbose: bool = True) -> str:
    """Build _build/liblp_san.so: the library with its host logic (argument
    checks, workspace layout, MGRIT schedule) compiled with AddressSanitizer and
    UndefinedBehaviorSanitizer; the kernel translation units are the ordinary
    objects (built first if missing)."""
    os.makedirs(os.path.join(OBJ, "san"), exist_ok=True)
    objs = []
    for src in SOURCES:
        if src in SAN_SOURCES:
            obj = os.path.join(OBJ, "san", os.path.splitext(src)[0] + ".o")
            flags = [f for f in FLAGS if f != "-O3"] + SAN_FLAGS
            cmd = [HIPCC, *flags, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed on {src} (sanitized):\n{r.stdout}\n{r.stderr}")
        else:
            obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
            if not os.path.exists(obj):
                obj = _compile(src)
        objs.append(obj)
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
           "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-shared-libasan", *objs, "-o", SAN_OUT]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {SAN_OUT}")
    return SAN_OUT


def build(verbose: bool = True) -> str:
    """Compile every source (always: this is the build check) and link liblp.so."""
    os.makedirs(OBJ, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--sanitize":
        build_sanitized()
    else:
        build()
    sys.exit(0)
